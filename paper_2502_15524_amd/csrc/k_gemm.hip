// bf16 GEMMs Y[m][n] = sum_k X[m][k] * W[n][k] on gfx950 MFMA with fused
// epilogues (residual add, SwiGLU, fp32 logits).
//
// Both operands are K-contiguous ([out][in] weights, token-major
// activations), so every MFMA operand fragment is one 16-byte load. The MFMA
// "A" operand is the weight tile (output features on MFMA rows) and "B" the
// activation tile (tokens on MFMA columns); each lane therefore ends up with
// 4 consecutive output features of one token and stores them as one 8-byte
// write.
//
// The weight matrix W [N][K] is stored in the tiled matrix format (1 KiB
// blocks of 8 rows x 64 k, chunk c of row r at position c ^ r, 64-column slabs
// contiguous), so both kernels read weights in long contiguous runs.
//
// Two kernels:
//  * gemm_ring   - prefill: BN x BM x 64 tiles copied straight into an LDS ring
//                  of NS stages, 4 waves, 16x16x32 bf16 MFMA, XCD-aware order.
//  * gemm_skinny - decode (M <= 64 tokens): HBM-bound weight streaming, 4
//                  waves split K inside a workgroup, reduced through LDS in a
//                  fixed order (deterministic).
#include "hs_device.h"
#include "hs_kernels.h"

#include <stdlib.h>

#include <string>

namespace hs {

// ---------------------------------------------------------------- epilogue

template <int EPI>
__device__ __forceinline__ void store4(const GemmArgs& a, int m, int f, const f32x4_v& v) {
  if (m >= a.M || f >= a.N) return;
  if constexpr (EPI == EPI_F32) {
    float4 o = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(static_cast<float*>(a.Y) + (int64_t)m * a.ldy + f) = o;
  } else {
    float r0 = v[0], r1 = v[1], r2 = v[2], r3 = v[3];
    if constexpr (EPI == EPI_RESID) {
      const uint2 rr = *reinterpret_cast<const uint2*>(a.R + (int64_t)m * a.ldr + f);
      r0 += lo_bf(rr.x); r1 += hi_bf(rr.x); r2 += lo_bf(rr.y); r3 += hi_bf(rr.y);
    }
    uint2 o;
    o.x = pack2bf(r0, r1);
    o.y = pack2bf(r2, r3);
    *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.Y) + (int64_t)m * a.ldy + f) = o;
  }
}

// gate tile g and up tile u hold the same 16 FFN columns; f is the output
// column (FFN index) of the lane's first value.
__device__ __forceinline__ void store_swiglu(const GemmArgs& a, int m, int f, const f32x4_v& g,
                                             const f32x4_v& u) {
  if (m >= a.M || f >= (a.N >> 1)) return;
  uint2 o;
  o.x = pack2bf(silu_f(g[0]) * u[0], silu_f(g[1]) * u[1]);
  o.y = pack2bf(silu_f(g[2]) * u[2], silu_f(g[3]) * u[3]);
  *reinterpret_cast<uint2*>(static_cast<bf16_t*>(a.Y) + (int64_t)m * a.ldy + f) = o;
}

// ------------------------------------ tiled, buffer loads into an LDS ring
//
// Operand tiles go global -> LDS with buffer_load_dwordx4 ... lds (no register
// staging): one instruction moves 64 lanes x 16 B of one operand into 1 KiB of
// LDS, lane L landing at byte 16 L (8 rows x 64 k). A weight block of the
// tiled format is exactly one such instruction (its chunks are already in the
// LDS order), and consecutive row blocks of one 64-k slab are adjacent in
// memory. Activations are row-major; the buffer resource ends at the last row,
// so rows past M read zeros and need no clamping (weight rows past N only feed
// outputs that are never stored). A lane's address is one 32-bit offset, the
// per-instruction and per-k-step parts are scalar. LDS rows are unpadded; the
// 16-byte chunks of a row are XOR-swizzled by the row index so the 16 rows of
// an MFMA fragment read hit different banks. NS stages form a ring: the
// loads for tile k + NS - 1 are in flight while tile k is multiplied, and a
// wave waits only for tile k + 1 before the workgroup barrier. The copies are
// issued from inline assembly so that the compiler neither tracks them nor
// inserts waits for them; this code waits explicitly (vmcnt) before each
// barrier. K is processed in 64-column slabs; when K % 64 != 0 the activation
// columns up to the next multiple of 64 must be zero (the weights are).

typedef int v4i_t __attribute__((ext_vector_type(4)));

constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data format

__device__ __forceinline__ v4i_t buf_rsrc(const void* p, uint64_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  const uint32_t n = bytes >= 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
  return v4i_t{(int)(uint32_t)a, (int)(uint32_t)((a >> 32) & 0xFFFFu), (int)n, kRsrcWord3};
}

// 64 lanes x 16 bytes from rsrc + voff + soff into LDS bytes [lds, lds + 1024)
__device__ __forceinline__ void dma16(v4i_t rsrc, int voff, int soff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :: "v"(voff), "s"(rsrc), "s"(__builtin_amdgcn_readfirstlane(soff)),
                  "s"(__builtin_amdgcn_readfirstlane(lds))
               : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <int BN, int BM, int BK, int NS>
struct RTile {
  static constexpr int CPR = BK / 8;           // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;         // rows per load instruction
  static constexpr int WN = BN / 2, WM = BM / 2, TN = WN / 16, TM = WM / 16;
  static constexpr int WI = BN / 4 / RPI, XI = BM / 4 / RPI;  // instructions per wave
  static constexpr int LPS = WI + XI;          // loads per stage per wave
  static constexpr int W_BYTES = BN * BK * 2, STAGE = (BN + BM) * BK * 2;
  static_assert(BK == 64, "weights come in 64-column slabs");
  static_assert(WI >= 1 && XI >= 1, "tile too small for 4 waves");
};

// position of chunk c of row r inside its row
template <int CPR>
__device__ __forceinline__ int chunk_pos(int r, int c) {
  if constexpr (CPR == 8) return c ^ (r & 7);
  else return c ^ ((r >> 1) & 3);
}

// Multiply one stage (BK/32 steps of 32 k). Fragment reads are software
// pipelined against the MFMAs and the order is pinned with scheduling group
// barriers: the A fragment of row tile i+1 is read while the TM MFMAs of row
// tile i run, and the B fragments of the next 32-k step are read during the
// last row tile of the current one.
template <int CPR>
__device__ __forceinline__ bf16x8_v lds_frag(const bf16_t* s, int r, int c) {
  return as_bf16x8(ld16(s + (r * CPR + chunk_pos<CPR>(r, c)) * 8));
}

template <int BN, int BM, int BK, int NS, int TN, int TM, typename Dma>
__device__ __forceinline__ void ring_stage(f32x4_v (&acc)[TN][TM], const bf16_t* sw,
                                           const bf16_t* sx, int wn, int wm, int fr, int g,
                                           Dma&& dma) {
  using T = RTile<BN, BM, BK, NS>;
  constexpr int CPR = T::CPR, KS = BK / 32;
  constexpr int MASK_MFMA = 0x008, MASK_DS_READ = 0x100;
  bf16x8_v b[2][TM];
  bf16x8_v a[2];
#pragma unroll
  for (int j = 0; j < TM; ++j) b[0][j] = lds_frag<CPR>(sx, wm * T::WM + j * 16 + fr, g);
  a[0] = lds_frag<CPR>(sw, wn * T::WN + fr, g);
  __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, TM + 1, 0);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int c = ks * 4 + g;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      const int cur = i & 1, nxt = cur ^ 1;
      dma(ks * TN + i);
      if (i + 1 < TN) {
        a[nxt] = lds_frag<CPR>(sw, wn * T::WN + (i + 1) * 16 + fr, c);
      } else if (ks + 1 < KS) {
#pragma unroll
        for (int j = 0; j < TM; ++j)
          b[(ks + 1) & 1][j] = lds_frag<CPR>(sx, wm * T::WM + j * 16 + fr, c + 4);
        a[nxt] = lds_frag<CPR>(sw, wn * T::WN + fr, c + 4);
      }
#pragma unroll
      for (int j = 0; j < TM; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[cur], b[ks & 1][j], acc[i][j], 0, 0, 0);
      if (i + 1 < TN) __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, 1, 0);
      else if (ks + 1 < KS) __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, TM + 1, 0);
      __builtin_amdgcn_sched_group_barrier(MASK_MFMA, TM, 0);
    }
  }
}

template <int BN, int BM, int BK, int NS, int WPE, int SPREAD, int EPI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
void gemm_ring(GemmArgs a) {
  using T = RTile<BN, BM, BK, NS>;
  constexpr int CPR = T::CPR, RPI = T::RPI, WN = T::WN, WM = T::WM, TN = T::TN, TM = T::TM;
  static_assert(EPI != EPI_SWIGLU || (WN % 32) == 0, "SwiGLU needs gate/up tile pairs");
  __shared__ __attribute__((aligned(1024))) char smem[NS * T::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1;
  const int tiles_m = (a.M + BM - 1) / BM;
  int bid = blockIdx.x;
  const int nb = gridDim.x;
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int n0 = (bid / tiles_m) * BN, m0 = (bid % tiles_m) * BM;

  const int kp = (a.K + 63) & ~63;
  const v4i_t rw = buf_rsrc(a.W, (uint64_t)a.N * kp * 2);
  const v4i_t rx = buf_rsrc(a.X, (uint64_t)a.M * a.ldx * 2);
  const int lrow = lane / CPR;
  const int lchunk = chunk_pos<CPR>(lrow, lane % CPR);  // row base is a multiple of RPI
  // weights: block (kt, n0/8 + wave * BN/32 + j) of the tiled format
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int vw = lane * 16;
  const int sw_base = (n0 / 8 + wave_u * (BN / 32)) * 1024, sw_step = 1024;
  const int sw_slab = (a.N / 8) * 1024;
  const int vx = ((m0 + wave * (BM / 4) + lrow) * (int)a.ldx + lchunk * 8) * 2;
  const int sx_step = RPI * (int)a.ldx * 2;
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) char*)smem;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t lds_w = lds0 + wave_s * (BN / 4) * BK * 2;
  const uint32_t lds_x = lds0 + T::W_BYTES + wave_s * (BM / 4) * BK * 2;

  // load instruction q of a stage: W rows first, then X rows
  auto issue_one = [&](int stage, int kt, int q) {
    const uint32_t so = stage * T::STAGE;
    if (q < T::WI) dma16(rw, vw, sw_base + kt * sw_slab + q * sw_step, lds_w + so + q * 1024);
    else dma16(rx, vx, (q - T::WI) * sx_step + kt * BK * 2, lds_x + so + (q - T::WI) * 1024);
  };
  auto issue = [&](int stage, int kt) {
#pragma unroll
    for (int q = 0; q < T::LPS; ++q) issue_one(stage, kt, q);
  };
  // spread the LPS loads of a stage over the TN * BK/32 row-tile steps
  constexpr int STEPS = TN * (BK / 32);
  auto issue_part = [&](int stage, int kt, int step) {
#pragma unroll
    for (int q = step * T::LPS / STEPS; q < (step + 1) * T::LPS / STEPS; ++q)
      issue_one(stage, kt, q);
  };

  f32x4_v acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, g = lane >> 4;
  const int nk = kp / BK;
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nk) issue(s, s);
  if (nk >= NS - 1) wait_vm<(NS - 2) * T::LPS>();
  else wait_vm<0>();
  wg_barrier();

  for (int kt = 0; kt < nk; ++kt) {
    const int stage = kt % NS;
    const bool more = kt + NS - 1 < nk;
    const bf16_t* sw = reinterpret_cast<const bf16_t*>(smem + stage * T::STAGE);
    const bf16_t* sx = reinterpret_cast<const bf16_t*>(smem + stage * T::STAGE + T::W_BYTES);
    // SPREAD: the next stage's loads are issued between MFMA groups (best with
    // one wave per SIMD); otherwise all at once before the stage's MFMAs.
    if (!SPREAD && more) issue((kt + NS - 1) % NS, kt + NS - 1);
    ring_stage<BN, BM, BK, NS>(acc, sw, sx, wn, wm, fr, g, [&](int step) {
      if (SPREAD && more) issue_part((kt + NS - 1) % NS, kt + NS - 1, step);
    });
    if (more) wait_vm<(NS - 2) * T::LPS>();
    else wait_vm<0>();
    wg_barrier();
  }

  const int fq = g * 4;
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = m0 + wm * WM + j * 16 + fr;
    if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
      for (int i = 0; i < TN; i += 2)
        store_swiglu(a, m, (n0 + wn * WN + i * 16) / 2 + fq, acc[i][j], acc[i + 1][j]);
    } else {
#pragma unroll
      for (int i = 0; i < TN; ++i) store4<EPI>(a, m, n0 + wn * WN + i * 16 + fq, acc[i][j]);
    }
  }
}

// ------------------------------------------------------------ skinny (decode)
//
// A workgroup owns 16 * NF weight rows and all M <= 64 tokens; its 4 waves
// split the 64-column slabs of K. For one slab, the rows' two (or four) 1 KiB
// blocks are adjacent, so a wave reads 2 KiB per 16 rows contiguously; lane
// (row fr, group g) takes chunk 4 ks + g of its row for the ks-th 32-k MFMA.

template <int NF, int MCH, int U, int EPI>
__global__ __launch_bounds__(256) void gemm_skinny(GemmArgs a) {
  static_assert(EPI != EPI_SWIGLU || (NF % 2) == 0, "SwiGLU needs gate/up tile pairs");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16 * NF;
  const int kp = (a.K + 63) & ~63;
  const int nslab = kp / 64;
  const int sq = (nslab + 3) / 4;  // slabs per wave
  const int sb = wave * sq, se = min(nslab, sb + sq);
  const int fr = lane & 15, g = lane >> 4;
  const int64_t slab_bytes = (int64_t)(a.N / 8) * 1024;

  const char* wrow[NF];
  bool wok[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int n = n0 + 16 * f + fr;
    wok[f] = n < a.N;
    wrow[f] = reinterpret_cast<const char*>(a.W) + (int64_t)(n / 8) * 1024 + (n % 8) * 128;
  }
  const int r8 = fr % 8;
  const bf16_t* xrow[MCH];
#pragma unroll
  for (int c = 0; c < MCH; ++c) {
    const int m = 16 * c + fr;
    xrow[c] = (m < a.M) ? a.X + (int64_t)m * a.ldx : nullptr;
  }

  f32x4_v acc[NF][MCH];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int c = 0; c < MCH; ++c) acc[f][c] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  for (int s0 = sb; s0 < se; s0 += U) {
    pack8 wv[NF][U][2], xv[MCH][U][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sl = s0 + u;
      const bool ok = sl < se;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int chunk = ks * 4 + g;
#pragma unroll
        for (int f = 0; f < NF; ++f)
          wv[f][u][ks] = (ok && wok[f])
                             ? ld16(wrow[f] + sl * slab_bytes + ((chunk ^ r8) * 16))
                             : zero8();
#pragma unroll
        for (int c = 0; c < MCH; ++c)
          xv[c][u][ks] = (ok && xrow[c]) ? ld16(xrow[c] + sl * 64 + chunk * 8) : zero8();
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
          for (int c = 0; c < MCH; ++c)
            acc[f][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(wv[f][u][ks]), as_bf16x8(xv[c][u][ks]), acc[f][c], 0, 0, 0);
  }

  __shared__ f32x4_v red[3][NF][MCH][64];
  if (wave > 0) {
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int c = 0; c < MCH; ++c) red[wave - 1][f][c][lane] = acc[f][c];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int c = 0; c < MCH; ++c) acc[f][c] += red[w][f][c][lane];

  const int fq = g * 4;
#pragma unroll
  for (int c = 0; c < MCH; ++c) {
    const int m = 16 * c + fr;
    if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
      for (int f = 0; f < NF; f += 2)
        store_swiglu(a, m, (n0 + 16 * f) / 2 + fq, acc[f][c], acc[f + 1][c]);
    } else {
#pragma unroll
      for (int f = 0; f < NF; ++f) store4<EPI>(a, m, n0 + 16 * f + fq, acc[f][c]);
    }
  }
}

// ------------------------------------------------------------------ launch

namespace {

template <int NF, int MCH, int U>
hipError_t dispatch_epi_skinny(const GemmArgs& a, int epi, hipStream_t s) {
  const int grid = (a.N + 16 * NF - 1) / (16 * NF);
  switch (epi) {
    case EPI_STORE:
      hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_STORE>), dim3(grid), dim3(256), 0, s, a);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_RESID>), dim3(grid), dim3(256), 0, s, a);
      break;
    case EPI_SWIGLU:
      if constexpr (NF % 2 == 0) {
        hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_SWIGLU>), dim3(grid), dim3(256), 0, s, a);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case EPI_F32:
      hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_F32>), dim3(grid), dim3(256), 0, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int BN, int BM, int BK, int NS, int WPE, int SPREAD>
hipError_t dispatch_epi_ring(const GemmArgs& a, int epi, hipStream_t s) {
  const int tiles = ((a.N + BN - 1) / BN) * ((a.M + BM - 1) / BM);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_ring<BN, BM, BK, NS, WPE, SPREAD, EPI_STORE>), dim3(tiles), dim3(256), 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_ring<BN, BM, BK, NS, WPE, SPREAD, EPI_RESID>), dim3(tiles), dim3(256), 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_ring<BN, BM, BK, NS, WPE, SPREAD, EPI_SWIGLU>), dim3(tiles), dim3(256), 0, s, a); break;
    case EPI_F32: hipLaunchKernelGGL((gemm_ring<BN, BM, BK, NS, WPE, SPREAD, EPI_F32>), dim3(tiles), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

const char* kEpiName[4] = {"store", "resid", "swiglu", "f32"};

}  // namespace

hipError_t gemm(const GemmArgs& a, int epi, hipStream_t s, LaunchInfo* info) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return hipErrorInvalidValue;
  if (epi < 0 || epi > 3) return hipErrorInvalidValue;
  const int64_t kp = (a.K + 63) / 64 * 64;
  if ((a.K % 8) || (a.N % 16) || (a.ldx % 8) || (a.ldy % 4)) return hipErrorInvalidValue;
  if ((a.K % 64) && a.ldx < kp) return hipErrorInvalidValue;
  if (epi == EPI_SWIGLU && (a.N % 32)) return hipErrorInvalidValue;
  if (epi == EPI_RESID && (!a.R || (a.ldr % 4))) return hipErrorInvalidValue;
  if (((uintptr_t)a.X | (uintptr_t)a.W | (uintptr_t)a.Y) & 15) return hipErrorInvalidValue;
  // 32-bit byte offsets in the buffer loads
  if ((uint64_t)a.N * kp * 2 >= (1ull << 31) || (uint64_t)a.M * a.ldx * 2 >= (1ull << 31))
    return hipErrorInvalidValue;

  static thread_local char name[64];
  const double flops = 2.0 * a.M * (double)a.N * a.K;
  const double out_cols = epi == EPI_SWIGLU ? a.N / 2 : a.N;
  const double out_bytes = (double)a.M * out_cols * (epi == EPI_F32 ? 4 : 2) *
                           (epi == EPI_RESID ? 2 : 1);
  const double bytes = 2.0 * ((double)a.M * a.K + (double)a.N * a.K) + out_bytes;
  hipError_t e;
  if (a.M <= 64) {
    const int mch = (a.M + 15) / 16;
    if (epi == EPI_SWIGLU) {
      switch (mch) {
        case 1: e = dispatch_epi_skinny<2, 1, 2>(a, epi, s); break;
        case 2: e = dispatch_epi_skinny<2, 2, 2>(a, epi, s); break;
        case 3: e = dispatch_epi_skinny<2, 3, 1>(a, epi, s); break;
        default: e = dispatch_epi_skinny<2, 4, 1>(a, epi, s); break;
      }
    } else {
      switch (mch) {
        case 1: e = dispatch_epi_skinny<1, 1, 4>(a, epi, s); break;
        case 2: e = dispatch_epi_skinny<1, 2, 2>(a, epi, s); break;
        case 3: e = dispatch_epi_skinny<1, 3, 2>(a, epi, s); break;
        default: e = dispatch_epi_skinny<1, 4, 1>(a, epi, s); break;
      }
    }
    snprintf(name, sizeof name, "gemm_skinny_%s", kEpiName[epi]);
  } else {
    // Tile choice; HS_GEMM_CFG forces one (tuning only).
    static const char* force = getenv("HS_GEMM_CFG");
    const long b256 = (long)((a.N + 255) / 256) * ((a.M + 255) / 256);
    const long t256x128 = (long)((a.N + 255) / 256) * ((a.M + 127) / 128);
    std::string cfg;
    if (force && *force) cfg = force;
    else if (b256 >= 256) cfg = "r256x256";       // large M: 1 wave / SIMD, 2 stages
    else if (t256x128 >= 160) cfg = "r256x128s3"; // mid-size: 3-stage ring
    else cfg = "r128x64s4";                       // few tiles: smaller ones, 4 stages
    if (cfg == "r256x256") e = dispatch_epi_ring<256, 256, 64, 2, 1, 1>(a, epi, s);
    else if (cfg == "r256x128s3") e = dispatch_epi_ring<256, 128, 64, 3, 1, 1>(a, epi, s);
    else if (cfg == "r128x128") e = dispatch_epi_ring<128, 128, 64, 2, 2, 0>(a, epi, s);
    else if (cfg == "r128x64") e = dispatch_epi_ring<128, 64, 64, 3, 2, 0>(a, epi, s);
    else e = dispatch_epi_ring<128, 64, 64, 4, 1, 1>(a, epi, s);
    snprintf(name, sizeof name, "gemm_%s_%s", cfg.c_str(), kEpiName[epi]);
  }
  if (info) {
    info->name = name;
    info->flops = flops;
    info->bytes = bytes;
  }
  return e;
}

}  // namespace hs
