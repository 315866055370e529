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
// Two kernels:
//  * gemm_tiled  - prefill: LDS double-buffered BN x BM x BK tiles, 4 waves,
//                  16x16x32 bf16 MFMA, XCD-aware tile order.
//  * gemm_skinny - decode (M <= 64 tokens): HBM-bound weight streaming, 4
//                  waves split K inside a workgroup, reduced through LDS in a
//                  fixed order (deterministic).
#include "hs_device.h"
#include "hs_kernels.h"

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

// ------------------------------------------------------------ tiled (prefill)

template <int BN, int BM, int BK, int WN, int WM, int EPI>
__global__ __launch_bounds__(64 * (BN / WN) * (BM / WM)) void gemm_tiled(GemmArgs a) {
  constexpr int NWN = BN / WN, NWM = BM / WM, NT = 64 * NWN * NWM;
  constexpr int TN = WN / 16, TM = WM / 16;
  constexpr int LK = BK + 8;  // padded LDS row (elements)
  constexpr int CPR = BK / 8; // 16-byte chunks per tile row
  constexpr int WCH = BN * CPR / NT, XCH = BM * CPR / NT;
  static_assert(BN * CPR % NT == 0 && BM * CPR % NT == 0, "tile/threads mismatch");
  static_assert(EPI != EPI_SWIGLU || (WN % 32) == 0, "SwiGLU needs gate/up tile pairs");

  __shared__ __attribute__((aligned(16))) bf16_t sW[2][BN * LK];
  __shared__ __attribute__((aligned(16))) bf16_t sX[2][BM * LK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave % NWN, wm = wave / NWN;

  const int tiles_m = (a.M + BM - 1) / BM;
  int bid = blockIdx.x;
  const int nb = gridDim.x;
  // Workgroups are dealt round-robin to the 8 XCDs; renumber so that each XCD
  // gets a contiguous range of tiles (tiles sharing a weight panel share L2).
  if ((nb & 7) == 0) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int n0 = (bid / tiles_m) * BN, m0 = (bid % tiles_m) * BM;

  f32x4_v acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4_v{0.f, 0.f, 0.f, 0.f};

  pack8 rw[WCH], rx[XCH];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      const int c = tid + i * NT, row = c / CPR, k = k0 + (c % CPR) * 8, n = n0 + row;
      rw[i] = (n < a.N && k < a.K) ? ld16(a.W + (int64_t)n * a.ldw + k) : zero8();
    }
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      const int c = tid + i * NT, row = c / CPR, k = k0 + (c % CPR) * 8, m = m0 + row;
      rx[i] = (m < a.M && k < a.K) ? ld16(a.X + (int64_t)m * a.ldx + k) : zero8();
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      const int c = tid + i * NT;
      st16(&sW[buf][(c / CPR) * LK + (c % CPR) * 8], rw[i]);
    }
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      const int c = tid + i * NT;
      st16(&sX[buf][(c / CPR) * LK + (c % CPR) * 8], rx[i]);
    }
  };

  const int nk = (a.K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int fr = lane & 15, kg = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const bf16_t* ws = sW[cur] + (wn * WN + fr) * LK + kg;
    const bf16_t* xs = sX[cur] + (wm * WM + fr) * LK + kg;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8_v af[TN], bf[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) af[i] = as_bf16x8(ld16(ws + i * 16 * LK + ks * 32));
#pragma unroll
      for (int j = 0; j < TM; ++j) bf[j] = as_bf16x8(ld16(xs + j * 16 * LK + ks * 32));
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  const int fq = (lane >> 4) * 4;
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

template <int NF, int MCH, int U, int EPI>
__global__ __launch_bounds__(256) void gemm_skinny(GemmArgs a) {
  static_assert(EPI != EPI_SWIGLU || (NF % 2) == 0, "SwiGLU needs gate/up tile pairs");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16 * NF;
  const int kq = ((a.K + 127) / 128) * 32;  // per-wave K range, multiple of 32
  const int kb = wave * kq, ke = min(a.K, kb + kq);
  const int fr = lane & 15, kg = (lane >> 4) * 8;

  const bf16_t* wrow[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int n = n0 + 16 * f + fr;
    wrow[f] = (n < a.N) ? a.W + (int64_t)n * a.ldw : nullptr;
  }
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

  for (int k0 = kb; k0 < ke; k0 += 32 * U) {
    pack8 wv[NF][U], xv[MCH][U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = k0 + 32 * u + kg;
      const bool ok = k < ke;
#pragma unroll
      for (int f = 0; f < NF; ++f) wv[f][u] = (ok && wrow[f]) ? ld16(wrow[f] + k) : zero8();
#pragma unroll
      for (int c = 0; c < MCH; ++c) xv[c][u] = (ok && xrow[c]) ? ld16(xrow[c] + k) : zero8();
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int c = 0; c < MCH; ++c)
          acc[f][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wv[f][u]),
                                                              as_bf16x8(xv[c][u]), acc[f][c],
                                                              0, 0, 0);
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

  const int fq = (lane >> 4) * 4;
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

template <int BN, int BM, int BK, int WN, int WM, int EPI>
hipError_t launch_tiled(const GemmArgs& a, hipStream_t s) {
  const int tiles = ((a.N + BN - 1) / BN) * ((a.M + BM - 1) / BM);
  constexpr int NT = 64 * (BN / WN) * (BM / WM);
  hipLaunchKernelGGL((gemm_tiled<BN, BM, BK, WN, WM, EPI>), dim3(tiles), dim3(NT), 0, s, a);
  return hipGetLastError();
}

template <int BN, int BM, int BK, int WN, int WM>
hipError_t dispatch_epi_tiled(const GemmArgs& a, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_STORE: return launch_tiled<BN, BM, BK, WN, WM, EPI_STORE>(a, s);
    case EPI_RESID: return launch_tiled<BN, BM, BK, WN, WM, EPI_RESID>(a, s);
    case EPI_SWIGLU: return launch_tiled<BN, BM, BK, WN, WM, EPI_SWIGLU>(a, s);
    case EPI_F32: return launch_tiled<BN, BM, BK, WN, WM, EPI_F32>(a, s);
  }
  return hipErrorInvalidValue;
}

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

const char* kEpiName[4] = {"store", "resid", "swiglu", "f32"};

}  // namespace

hipError_t gemm(const GemmArgs& a, int epi, hipStream_t s, LaunchInfo* info) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return hipErrorInvalidValue;
  if (epi < 0 || epi > 3) return hipErrorInvalidValue;
  if ((a.K % 8) || (a.N % 16) || (a.ldx % 8) || (a.ldw % 8) || (a.ldy % 4)) return hipErrorInvalidValue;
  if (epi == EPI_SWIGLU && (a.N % 32)) return hipErrorInvalidValue;
  if (epi == EPI_RESID && (!a.R || (a.ldr % 4))) return hipErrorInvalidValue;
  if (((uintptr_t)a.X | (uintptr_t)a.W) & 15) return hipErrorInvalidValue;
  if ((uintptr_t)a.Y & 15) return hipErrorInvalidValue;

  static thread_local char name[64];
  const double flops = 2.0 * a.M * (double)a.N * a.K;
  const double out_cols = epi == EPI_SWIGLU ? a.N / 2 : a.N;
  const double out_bytes = (double)a.M * out_cols * (epi == EPI_F32 ? 4 : 2) *
                           (epi == EPI_RESID ? 2 : 1);
  const double bytes = 2.0 * ((double)a.M * a.K + (double)a.N * a.K) + out_bytes;
  hipError_t e;
  if (a.M <= 64) {
    const int mch = (a.M + 15) / 16;
    const bool two = (epi == EPI_SWIGLU);
    if (two) {
      switch (mch) {
        case 1: e = dispatch_epi_skinny<2, 1, 4>(a, epi, s); break;
        case 2: e = dispatch_epi_skinny<2, 2, 4>(a, epi, s); break;
        case 3: e = dispatch_epi_skinny<2, 3, 2>(a, epi, s); break;
        default: e = dispatch_epi_skinny<2, 4, 2>(a, epi, s); break;
      }
    } else {
      switch (mch) {
        case 1: e = dispatch_epi_skinny<1, 1, 8>(a, epi, s); break;
        case 2: e = dispatch_epi_skinny<1, 2, 4>(a, epi, s); break;
        case 3: e = dispatch_epi_skinny<1, 3, 4>(a, epi, s); break;
        default: e = dispatch_epi_skinny<1, 4, 2>(a, epi, s); break;
      }
    }
    snprintf(name, sizeof name, "gemm_skinny_%s", kEpiName[epi]);
  } else {
    const long t256 = (long)((a.N + 255) / 256) * ((a.M + 127) / 128);
    const long t128 = (long)((a.N + 127) / 128) * ((a.M + 127) / 128);
    const long t64 = (long)((a.N + 127) / 128) * ((a.M + 63) / 64);
    if (t256 >= 256) {
      e = dispatch_epi_tiled<256, 128, 64, 128, 64>(a, epi, s);
      snprintf(name, sizeof name, "gemm_256x128_%s", kEpiName[epi]);
    } else if (t128 >= 256) {
      e = dispatch_epi_tiled<128, 128, 64, 64, 64>(a, epi, s);
      snprintf(name, sizeof name, "gemm_128x128_%s", kEpiName[epi]);
    } else if (t64 >= 128) {
      e = dispatch_epi_tiled<128, 64, 64, 64, 32>(a, epi, s);
      snprintf(name, sizeof name, "gemm_128x64_%s", kEpiName[epi]);
    } else {
      e = dispatch_epi_tiled<64, 64, 64, 32, 32>(a, epi, s);
      snprintf(name, sizeof name, "gemm_64x64_%s", kEpiName[epi]);
    }
  }
  if (info) {
    info->name = name;
    info->flops = flops;
    info->bytes = bytes;
  }
  return e;
}

}  // namespace hs
