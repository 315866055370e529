// Memory-bound helpers of the stage forward pass: embedding gather, RMSNorm,
// rotary embedding with paged KV append, greedy argmax and the KV block copy
// used by export, import and merge.
#include "hs_device.h"
#include "hs_kernels.h"

namespace hs {

// ------------------------------------------------------------ call metadata
//
// A stage call's metadata (positions, slots, tiles, block tables) is written
// by the host into pinned memory and pulled into device memory by this kernel
// at the start of the call. A kernel launch follows the previous kernel
// directly, whereas a copy command waits behind a fence of its own (about
// 5.5 us of idle GPU on MI355X). The loads are system-coherent (sc0 sc1), so
// they see what the host wrote before the launch, never a cached copy of an
// earlier call's values.

// Workgroups [0, b0) copy the first segment, the rest the second.
__global__ __launch_bounds__(256) void meta_pull_kernel(const int32_t* h0, int32_t* d0,
                                                        int64_t n0, const int32_t* h1,
                                                        int32_t* d1, int64_t n1, int b0) {
  const bool first = (int)blockIdx.x < b0;
  const int64_t i = (int64_t)(first ? blockIdx.x : blockIdx.x - b0) * 256 + threadIdx.x;
  const int64_t n16 = first ? n0 : n1;
  if (i >= n16) return;
  typedef unsigned u32x4_v __attribute__((ext_vector_type(4)));
  constexpr int kSystem = 1 | 16;  // sc0 | sc1
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(first ? h0 : h1), 0, (int)(n16 * 16), 0x00020000);
  const u32x4_v v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(i * 16), 0, kSystem);
  *reinterpret_cast<u32x4_v*>((first ? d0 : d1) + i * 4) = v;
}

hipError_t meta_pull(const int32_t* host, int32_t* dev, int64_t n, hipStream_t s,
                     const int32_t* host2, int32_t* dev2, int64_t n2) {
  if (n < 0 || n2 < 0 || (n % 4) || (n2 % 4) || n * 4 >= (1ll << 31) || n2 * 4 >= (1ll << 31) ||
      (n && (((uintptr_t)host | (uintptr_t)dev) & 15)) ||
      (n2 && (((uintptr_t)host2 | (uintptr_t)dev2) & 15)))
    return hipErrorInvalidValue;
  const int b0 = (int)((n / 4 + 255) / 256), b1 = (int)((n2 / 4 + 255) / 256);
  if (b0 + b1 == 0) return hipSuccess;
  hipLaunchKernelGGL(meta_pull_kernel, dim3((unsigned)(b0 + b1)), dim3(256), 0, s, host, dev,
                     n / 4, host2, dev2, n2 / 4, b0);
  return hipGetLastError();
}

// ---------------------------------------------------------------- embedding

__global__ __launch_bounds__(256) void embed_kernel(const int32_t* tok, const bf16_t* E, int vocab,
                                                    int hidden, bf16_t* out) {
  const int t = blockIdx.x;
  const int id = tok[t];
  const bool ok = id >= 0 && id < vocab;  // out-of-range ids give a zero row
  const int chunks = hidden / 8;
  for (int c = threadIdx.x; c < chunks; c += blockDim.x) {
    const pack8 v = ok ? ld16(E + (int64_t)id * hidden + c * 8) : zero8();
    st16(out + (int64_t)t * hidden + c * 8, v);
  }
}

hipError_t embed(const int32_t* tok, const bf16_t* E, int vocab, int hidden, int n_tok,
                 bf16_t* out, hipStream_t s, LaunchInfo* info) {
  if (n_tok <= 0) return hipSuccess;
  if (hidden % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_kernel, dim3(n_tok), dim3(256), 0, s, tok, E, vocab, hidden, out);
  if (info) *info = LaunchInfo{"embed", 0, 4.0 * n_tok * (double)hidden};
  return hipGetLastError();
}

// ------------------------------------------------------------------ RMSNorm

// One workgroup per row; each thread keeps up to 4 chunks of 8 values and
// loads the gain's chunks together with the row's (one memory round trip per
// row: the gain does not wait for the reduction).
__global__ __launch_bounds__(256) void rmsnorm_kernel(const bf16_t* x, int64_t ldx,
                                                      const int32_t* rows, int hidden,
                                                      const bf16_t* gain, float eps, bf16_t* out,
                                                      int64_t ldo) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const int src = rows ? rows[r] : r;
  const bf16_t* xr = x + (int64_t)src * ldx;
  const int chunks = hidden / 8;
  pack8 xv[4], gv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = threadIdx.x + i * 256;
    if (c < chunks) {
      xv[i] = ld16(xr + c * 8);
      gv[i] = ld16(gain + c * 8);
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (threadIdx.x + i * 256 < chunks) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = lo_bf(xv[i].w[e]), hi = hi_bf(xv[i].w[e]);
        ss += lo * lo;
        ss += hi * hi;
      }
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / sqrtf(tot / (float)hidden + eps);
  bf16_t* orow = out + (int64_t)r * ldo;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = threadIdx.x + i * 256;
    if (c < chunks) {
      pack8 o;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        o.w[e] = pack2bf(lo_bf(xv[i].w[e]) * inv * lo_bf(gv[i].w[e]),
                         hi_bf(xv[i].w[e]) * inv * hi_bf(gv[i].w[e]));
      st16(orow + c * 8, o);
    }
  }
}

hipError_t rmsnorm(const bf16_t* x, int64_t ldx, const int32_t* rows, int n_rows, int hidden,
                   const bf16_t* g, float eps, bf16_t* out, int64_t ldo, hipStream_t s,
                   LaunchInfo* info) {
  if (n_rows <= 0) return hipSuccess;
  if ((hidden % 8) || hidden > 8192 || (ldx % 8) || (ldo % 8)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(n_rows), dim3(256), 0, s, x, ldx, rows, hidden, g, eps,
                     out, ldo);
  if (info) *info = LaunchInfo{"rmsnorm", 0, 4.0 * n_rows * (double)hidden};
  return hipGetLastError();
}

// --------------------------------------------------- RoPE + paged KV append
//
// Work item = 4 consecutive rotation pairs (i, i + D/2), i = 4j .. 4j + 3, of
// one q or k head of one token (8-byte loads and stores of each half), or one
// 16-byte chunk of one v head. q and k are rotated in place (rotate-half,
// angle pos * base^(-2i/D) from the table); the rotated k and the v of each
// KV head are also written to the token's slot in the paged pool. Grid:
// (tokens, work items / 256).

__global__ __launch_bounds__(256) void rope_kv_kernel(RopeKvArgs a) {
  const int t = blockIdx.x;
  const int half = a.D / 2, q4 = half / 4;          // 4-pair groups per head
  const int n_rot = (a.n_heads + a.n_kv_heads) * q4;
  const int n_v = a.n_kv_heads * (a.D / 8);
  const int i = blockIdx.y * 256 + threadIdx.x;
  if (i >= n_rot + n_v) return;
  const int pos = a.pos[t];
  const int slot = a.slot[t];
  bf16_t* row = a.qkv + (int64_t)t * a.ld;
  const int64_t blk_base = slot >= 0 ? (int64_t)(slot >> 4) * 2 * a.n_kv_heads * 16 * a.D : 0;
  const int off = slot & 15;
  if (i < n_rot) {
    const int head = i / q4, j = (i % q4) * 4;
    bf16_t* hp = row + head * a.D;
    const uint2 lo = *reinterpret_cast<const uint2*>(hp + j);
    const uint2 hi = *reinterpret_cast<const uint2*>(hp + j + half);
    const float4 c = *reinterpret_cast<const float4*>(a.cos_t + (int64_t)pos * half + j);
    const float4 sn = *reinterpret_cast<const float4*>(a.sin_t + (int64_t)pos * half + j);
    const float x1[4] = {lo_bf(lo.x), hi_bf(lo.x), lo_bf(lo.y), hi_bf(lo.y)};
    const float x2[4] = {lo_bf(hi.x), hi_bf(hi.x), lo_bf(hi.y), hi_bf(hi.y)};
    const float cc[4] = {c.x, c.y, c.z, c.w}, ss[4] = {sn.x, sn.y, sn.z, sn.w};
    float y1[4], y2[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y1[e] = rope_first(x1[e], x2[e], cc[e], ss[e]);
      y2[e] = rope_second(x1[e], x2[e], cc[e], ss[e]);
    }
    const uint2 o1 = make_uint2(pack2bf(y1[0], y1[1]), pack2bf(y1[2], y1[3]));
    const uint2 o2 = make_uint2(pack2bf(y2[0], y2[1]), pack2bf(y2[2], y2[3]));
    *reinterpret_cast<uint2*>(hp + j) = o1;
    *reinterpret_cast<uint2*>(hp + j + half) = o2;
    if (head >= a.n_heads && slot >= 0) {
      bf16_t* kp = a.pool + blk_base + (int64_t)(head - a.n_heads) * 16 * a.D + off * a.D;
      *reinterpret_cast<uint2*>(kp + j) = o1;
      *reinterpret_cast<uint2*>(kp + j + half) = o2;
    }
  } else if (slot >= 0) {
    const int v = i - n_rot, kh = v / (a.D / 8), c = v % (a.D / 8);
    const pack8 x = ld16(row + (a.n_heads + a.n_kv_heads + kh) * a.D + c * 8);
    st16(a.pool + blk_base + ((int64_t)a.n_kv_heads + kh) * 16 * a.D + off * a.D + c * 8, x);
  }
}

hipError_t rope_kv(const RopeKvArgs& a, hipStream_t s, LaunchInfo* info) {
  if (a.T <= 0) return hipSuccess;
  if ((a.D % 16) || (a.ld % 8)) return hipErrorInvalidValue;
  const int items = (a.n_heads + a.n_kv_heads) * (a.D / 8) + a.n_kv_heads * (a.D / 8);
  hipLaunchKernelGGL(rope_kv_kernel, dim3(a.T, (items + 255) / 256), dim3(256), 0, s, a);
  if (info) {
    const double row = (double)(a.n_heads + 2 * a.n_kv_heads) * a.D * 2;
    *info = LaunchInfo{"rope_kv", 0, a.T * (row + (double)(a.n_heads + a.n_kv_heads) * a.D * 2 +
                                            2.0 * a.n_kv_heads * a.D * 2)};
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------- argmax

__device__ __forceinline__ void better(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

// Two passes: workgroups of the first take 4096-column chunks of a row (four
// 16-byte loads per thread, all in flight together) and leave the chunk's
// best (value, index); the second reduces a row's chunks in chunk order.
// Ties go to the lowest index in both, so the result is the row's lowest
// index of the maximum.
constexpr int kArgmaxChunk = 4096;

__device__ __forceinline__ void wave_best(float& bv, int& bi) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(bv, o, 64);
    const int i2 = __shfl_xor(bi, o, 64);
    better(bv, bi, v2, i2);
  }
}

__global__ __launch_bounds__(256) void argmax_chunk_kernel(const float* logits, int n_cols,
                                                           int n_chunks, int32_t* part) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int chunk = blockIdx.x, row = blockIdx.y;
  const float* r = logits + (int64_t)row * n_cols;
  const int c0 = chunk * kArgmaxChunk + threadIdx.x * 4;
  float4 v[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = c0 + u * 1024;
    v[u] = c < n_cols ? *reinterpret_cast<const float4*>(r + c)
                      : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  }
  float bv = -INFINITY;
  int bi = 0x7FFFFFFF;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int c = c0 + u * 1024;
    if (c < n_cols) {
      better(bv, bi, v[u].x, c);
      better(bv, bi, v[u].y, c + 1);
      better(bv, bi, v[u].z, c + 2);
      better(bv, bi, v[u].w, c + 3);
    }
  }
  wave_best(bv, bi);
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = bv;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) better(bv, bi, sv[w], si[w]);
    int32_t* o = part + ((int64_t)row * n_chunks + chunk) * 2;
    o[0] = __float_as_int(bv);
    o[1] = bi;
  }
}

__global__ __launch_bounds__(64) void argmax_final_kernel(const int32_t* part, int n_chunks,
                                                          int32_t* out) {
  const int row = blockIdx.x;
  float bv = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int c = threadIdx.x; c < n_chunks; c += 64) {
    const int32_t* p = part + ((int64_t)row * n_chunks + c) * 2;
    better(bv, bi, __int_as_float(p[0]), p[1]);
  }
  wave_best(bv, bi);
  if (threadIdx.x == 0) out[row] = bi;
}

int argmax_chunks(int n_cols) { return (n_cols + kArgmaxChunk - 1) / kArgmaxChunk; }

hipError_t argmax_rows(const float* logits, int n_rows, int n_cols, int32_t* part, int32_t* out,
                       hipStream_t s, LaunchInfo* info) {
  if (n_rows <= 0) return hipSuccess;
  if (n_cols <= 0 || (n_cols % 4) || !part) return hipErrorInvalidValue;
  const int nc = argmax_chunks(n_cols);
  hipLaunchKernelGGL(argmax_chunk_kernel, dim3(nc, n_rows), dim3(256), 0, s, logits, n_cols, nc,
                     part);
  hipLaunchKernelGGL(argmax_final_kernel, dim3(n_rows), dim3(64), 0, s, part, nc, out);
  if (info) *info = LaunchInfo{"argmax", 0, 4.0 * n_rows * (double)n_cols};
  return hipGetLastError();
}

// ------------------------------------------------------------------ KV copy
//
// A unit is one KV block of one layer: the K block [n_kv][16][D] followed by
// the V block, contiguous both in the pools and in the blob. Each workgroup
// copies up to 16 KiB of one unit: four 16-byte loads per thread issued
// together, then the four stores. Row r of a unit (D * 2 bytes, a power of
// two) holds token slot r % 16.


typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

template <int PER, bool NT>
__global__ __launch_bounds__(256) void kv_copy_kernel(const uint64_t* src, const uint64_t* dst,
                                                      const int32_t* valid, int64_t unit_bytes,
                                                      int row_shift, int zero_tail) {
  const int u = blockIdx.x;
  const char* s = reinterpret_cast<const char*>(src[u]);
  char* d = reinterpret_cast<char*>(dst[u]);
  const int v = zero_tail ? valid[u] : 16;
  const int64_t begin = (int64_t)blockIdx.y * (PER * 4096) + threadIdx.x * 16;
  u32x4_t x[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int64_t o = begin + k * 4096;
    const int slot = (int)((o >> row_shift) & 15);
    const u32x4_t* p = reinterpret_cast<const u32x4_t*>(s + o);
    if (o < unit_bytes && slot < v) x[k] = NT ? __builtin_nontemporal_load(p) : *p;
    else x[k] = u32x4_t{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int64_t o = begin + k * 4096;
    u32x4_t* p = reinterpret_cast<u32x4_t*>(d + o);
    if (o < unit_bytes) {
      if (NT) __builtin_nontemporal_store(x[k], p);
      else *p = x[k];
    }
  }
}

hipError_t kv_copy(const uint64_t* src, const uint64_t* dst, const int32_t* valid, int n_units,
                   int64_t unit_bytes, int D, int zero_tail, hipStream_t s, LaunchInfo* info) {
  if (n_units <= 0) return hipSuccess;
  if ((unit_bytes % 16) || (D != 64 && D != 128)) return hipErrorInvalidValue;
  const int row_shift = D == 128 ? 8 : 7;
  // 16 KiB per workgroup, streamed with non-temporal loads and stores (each
  // byte is read once and written once): 4.74 TB/s exporting 2.46 GB on
  // MI355X, where a plain device copy of the same bytes runs at 5.0 TB/s
  constexpr int kPer = 4;
  const int parts = (int)((unit_bytes + kPer * 4096 - 1) / (kPer * 4096));
  hipLaunchKernelGGL((kv_copy_kernel<kPer, true>), dim3(n_units, parts), dim3(256), 0, s, src, dst,
                     valid, unit_bytes, row_shift, zero_tail);
  if (info) *info = LaunchInfo{"kv_copy", 0, 2.0 * n_units * (double)unit_bytes};
  return hipGetLastError();
}

}  // namespace hs
