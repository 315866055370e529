// Device-side helpers shared by the engine's HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // raw bfloat16 bits
typedef __bf16 bf16x8_v __attribute__((ext_vector_type(8)));
typedef float f32x4_v __attribute__((ext_vector_type(4)));
typedef float f32x16_v __attribute__((ext_vector_type(16)));

// 16 bytes = 8 bf16 values.
struct alignas(16) pack8 {
  uint32_t w[4];
};

__device__ __forceinline__ float bf2f(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bf16, round to nearest even (finite inputs).
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

__device__ __forceinline__ uint32_t pack2bf(float lo, float hi) {
  return static_cast<uint32_t>(f2bf(lo)) | (static_cast<uint32_t>(f2bf(hi)) << 16);
}

__device__ __forceinline__ float lo_bf(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ pack8 ld16(const void* p) {
  return *reinterpret_cast<const pack8*>(p);
}
// 16 bytes read once per call (weights, cached keys and values): a
// non-temporal load
__device__ __forceinline__ pack8 ld16_nt(const void* p) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  pack8 r;
  r.w[0] = v[0];
  r.w[1] = v[1];
  r.w[2] = v[2];
  r.w[3] = v[3];
  return r;
}
__device__ __forceinline__ void st16(void* p, const pack8& v) {
  *reinterpret_cast<pack8*>(p) = v;
}
__device__ __forceinline__ pack8 zero8() {
  pack8 z;
  z.w[0] = z.w[1] = z.w[2] = z.w[3] = 0u;
  return z;
}

__device__ __forceinline__ bf16x8_v as_bf16x8(const pack8& v) {
  return __builtin_bit_cast(bf16x8_v, v);
}

// 2^x on the hardware exp unit.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float silu_f(float g) {
  // g * sigmoid(g), with e^-g = 2^(-g log2 e)
  return g / (1.0f + fast_exp2(-g * 1.4426950408889634f));
}

// Rotate-half RoPE of one pair: x1 at index i of a head's first half, x2 at
// i + D/2, angle with cosine c and sine s. Every kernel that rotates uses
// these two (with explicit fused multiply-adds), so they all round alike.
__device__ __forceinline__ float rope_first(float x1, float x2, float c, float s) {
  return fmaf(x1, c, -(x2 * s));
}
__device__ __forceinline__ float rope_second(float x1, float x2, float c, float s) {
  return fmaf(x2, c, x1 * s);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
