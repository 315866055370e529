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
//                  of NS stages, 8 waves, 16x16x32 bf16 MFMA, XCD-aware order.
//  * gemm_skinny - decode (M <= 64 tokens): HBM-bound weight streaming, 2,
//                  4 or 8 waves split K inside a workgroup, reduced through
//                  LDS in a fixed order (deterministic).
#include "hs_device.h"
#include "hs_kernels.h"

#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>

#include <string>

namespace hs {

// ---------------------------------------------------------------- epilogue

// Output column (head order) of column n of a QKV projection whose q and k
// rows are stored head-interleaved: inside a head, the 32-row group p holds
// rows 16p .. 16p + 15 of the first half, then the same rows of the second.
__device__ __forceinline__ int qk_col(const GemmArgs& a, int n) {
  if (n >= a.rope_q_cols + a.rope_kv_cols) return n;
  const int d = n & (a.rope_d - 1);
  return (n - d) + ((d >> 4) & 1) * (a.rope_d >> 1) + (d >> 5) * 16 + (d & 15);
}

template <int EPI>
__device__ __forceinline__ void store4(const GemmArgs& a, int m, int f, const f32x4_v& v) {
  if (m >= a.M || f >= a.N) return;
  if constexpr (EPI == EPI_STORE) f = qk_col(a, f);
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

// QKV projection with RoPE and KV append. n is the (stored-order) column of
// x1's first value, a multiple of 4 inside the first 16 rows of a 32-row
// pair; x2 holds the pair's other 16 rows. In the q and k heads these are
// RoPE partners (rotation index i and i + D/2); in the v heads two adjacent
// 16-column groups. Values are rounded to bf16 before the rotation, as a
// separate rotation pass reading the stored projection would see them.

// rotation index of column n (< rope_q_cols + rope_kv_cols) and its table offset
__device__ __forceinline__ int64_t rope_tab_off(const GemmArgs& a, int pos, int n) {
  const int d = n & (a.rope_d - 1);
  return (int64_t)pos * (a.rope_d >> 1) + (d >> 5) * 16 + (d & 15);
}

// cv, sv: cos and sin at rope_tab_off(a, pos, n) (unused for v columns)
__device__ __forceinline__ void store_qkv_rope(const GemmArgs& a, int m, int slot, int n,
                                               const f32x4_v& x1, const f32x4_v& x2,
                                               const float4& cv, const float4& sv) {
  if (m >= a.M || n >= a.N) return;
  const int D = a.rope_d, half = D >> 1;
  uint2 o1, o2;
  o1.x = pack2bf(x1[0], x1[1]);
  o1.y = pack2bf(x1[2], x1[3]);
  o2.x = pack2bf(x2[0], x2[1]);
  o2.y = pack2bf(x2[2], x2[3]);
  int c1, c2;  // output columns of x1 and x2
  if (n < a.rope_q_cols + a.rope_kv_cols) {
    const int d = n & (D - 1);
    c1 = (n - d) + (d >> 5) * 16 + (d & 15);
    c2 = c1 + half;
    const float cc[4] = {cv.x, cv.y, cv.z, cv.w}, ss[4] = {sv.x, sv.y, sv.z, sv.w};
    const float p1[4] = {lo_bf(o1.x), hi_bf(o1.x), lo_bf(o1.y), hi_bf(o1.y)};
    const float p2[4] = {lo_bf(o2.x), hi_bf(o2.x), lo_bf(o2.y), hi_bf(o2.y)};
    float y1[4], y2[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y1[e] = rope_first(p1[e], p2[e], cc[e], ss[e]);
      y2[e] = rope_second(p1[e], p2[e], cc[e], ss[e]);
    }
    o1 = make_uint2(pack2bf(y1[0], y1[1]), pack2bf(y1[2], y1[3]));
    o2 = make_uint2(pack2bf(y2[0], y2[1]), pack2bf(y2[2], y2[3]));
  } else {
    c1 = n;
    c2 = n + 16;
  }
  bf16_t* row = static_cast<bf16_t*>(a.Y) + (int64_t)m * a.ldy;
  *reinterpret_cast<uint2*>(row + c1) = o1;
  *reinterpret_cast<uint2*>(row + c2) = o2;
  if (slot >= 0 && n >= a.rope_q_cols) {
    // k head kh -> pool part 0, v head kh -> part 1 of the token's block
    const int n_kv = a.rope_kv_cols / D;
    const int kv = c1 - a.rope_q_cols;  // column inside the k (then v) heads
    const int kh = kv / D;              // 0 .. 2 n_kv - 1: k heads, then v heads
    bf16_t* dst = a.rope_pool + (int64_t)(slot >> 4) * 2 * n_kv * 16 * D +
                  ((int64_t)kh * 16 + (slot & 15)) * D + (kv - kh * D);
    *reinterpret_cast<uint2*>(dst) = o1;
    *reinterpret_cast<uint2*>(dst + (c2 - c1)) = o2;
  }
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

// NW waves per workgroup as 2 x NW/2: two wave columns over the BN weight
// rows, NW/2 wave rows over the BM tokens.
template <int BN, int BM, int BK, int NS, int NW = 4>
struct RTile {
  static constexpr int CPR = BK / 8;           // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;         // rows per load instruction
  static constexpr int WN = BN / 2, WM = BM / (NW / 2), TN = WN / 16, TM = WM / 16;
  static constexpr int WI = BN / NW / RPI, XI = BM / NW / RPI;  // instructions per wave
  static constexpr int LPS = WI + XI;          // loads per stage per wave
  static constexpr int W_BYTES = BN * BK * 2, STAGE = (BN + BM) * BK * 2;
  static_assert(BK == 64, "weights come in 64-column slabs");
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(WI >= 1 && XI >= 1 && TM >= 1, "tile too small for the waves");
};

// position of chunk c of row r inside its row
template <int CPR>
__device__ __forceinline__ int chunk_pos(int r, int c) {
  if constexpr (CPR == 8) return c ^ (r & 7);
  else return c ^ ((r >> 1) & 3);
}

// Multiply one stage (BK/32 steps of 32 k). Fragment reads are software
// pipelined against the MFMAs and the order is pinned with scheduling group
// barriers: the A fragment of row tile i + PD is read while the TM MFMAs of
// row tile i run, and the B fragments of the next 32-k step are read with the
// first A fragment that needs them. The last row tile of a stage is deferred
// past the workgroup barrier: it runs while the next stage's first fragments
// come from LDS (its operands are already in registers).
template <int CPR>
__device__ __forceinline__ bf16x8_v lds_frag(const bf16_t* s, int r, int c) {
  return as_bf16x8(ld16(s + (r * CPR + chunk_pos<CPR>(r, c)) * 8));
}

// How many row tiles ahead of its MFMAs a wave reads the A fragments: three
// for the 4- and 6-row-tile wave tiles (128 x 128 and 192-row tiles; 512-token
// 7B shapes, MI355X: gate/up 96.6 -> 94.0 us, QKV 55.8 -> 53.8, o 29.3 ->
// 28.2), one for the 8-row-tile ones of 256-row tiles (three made 8192-token
// launches 1-4 % slower). The fragments and MFMAs are the same either way.
template <int TN>
constexpr int ring_pd() {
  return (TN == 4 || TN == 6) ? 3 : 1;
}

template <int BN, int BM, int BK, int NS, int NW, int TN, int TM, int PD, typename Dma>
__device__ __forceinline__ void ring_stage(f32x4_v (&acc)[TN][TM], bf16x8_v (&a)[PD + 1],
                                           bf16x8_v (&b)[2][TM], const bf16_t* sw,
                                           const bf16_t* sx, int wn, int wm, int fr, int g,
                                           bool pending, Dma&& dma) {
  using T = RTile<BN, BM, BK, NS, NW>;
  constexpr int CPR = T::CPR, KS = BK / 32, NT = TN * KS;
  constexpr int MASK_MFMA = 0x008, MASK_DS_READ = 0x100;
  // 256 x 256 tiles: a wave runs its MFMA groups at raised priority, so the
  // SIMD's other wave issues its LDS reads and loads in between instead of
  // competing with them (8192 tokens, MI355X: gate/up 1155-1162 -> 1107-1113
  // us, down 580 -> 562; the smaller tiles gained nothing)
  constexpr bool PRIO = BN == 256 && BM == 256 && NW == 8;
  // row tile t of the stage (t = ks TN + i) uses A slot t mod (PD + 1); the
  // deferred last one must not share a slot with the next stage's first PD
  static_assert(KS == 2 && NT % (PD + 1) == 0, "A fragment slots");
  constexpr int LAST = (NT - 1) % (PD + 1);
  auto read_a = [&](int t) {
    a[t % (PD + 1)] = lds_frag<CPR>(sw, wn * T::WN + (t % TN) * 16 + fr, (t / TN) * 4 + g);
  };
#pragma unroll
  for (int j = 0; j < TM; ++j) b[0][j] = lds_frag<CPR>(sx, wm * T::WM + j * 16 + fr, g);
#pragma unroll
  for (int t = 0; t < PD; ++t) read_a(t);
  __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, TM + PD, 0);
  // the previous stage's last row tile (operands in registers) runs while
  // this stage's first fragments are on their way from LDS
  if (pending) {
#pragma unroll
    for (int j = 0; j < TM; ++j)
      acc[TN - 1][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[LAST], b[1][j], acc[TN - 1][j], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(MASK_MFMA, TM, 0);
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int ks = t / TN, i = t % TN;
    dma(t);
    // A of row tile t + PD; the B fragments of the next 32-k step together
    // with the A fragment that first needs them
    const bool ra = t + PD < NT, rb = ks + 1 < KS && i == TN - PD;
    if (ra) read_a(t + PD);
    if (rb) {
#pragma unroll
      for (int j = 0; j < TM; ++j)
        b[(ks + 1) & 1][j] = lds_frag<CPR>(sx, wm * T::WM + j * 16 + fr, (ks + 1) * 4 + g);
    }
    if (t == NT - 1) break;  // deferred to the next stage (or the end)
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int j = 0; j < TM; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t % (PD + 1)], b[ks & 1][j], acc[i][j], 0, 0, 0);
    if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
    if (ra && rb) __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, TM + 1, 0);
    else if (ra) __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, 1, 0);
    else if (rb) __builtin_amdgcn_sched_group_barrier(MASK_DS_READ, TM, 0);
    __builtin_amdgcn_sched_group_barrier(MASK_MFMA, TM, 0);
  }
}

// Tile schedule. Output tiles are numbered in groups of `group_n` column
// tiles (weight rows) by all row tiles (tokens), column tile fastest, so the
// workgroups that run together on one XCD share weight and activation slabs
// in its L2. A data-parallel launch runs one whole tile per workgroup. A
// stream-K launch gives each of its G workgroups an equal contiguous share of
// the (tile, 64-k step) iteration space; a tile whose k range is split
// between workgroups is finished by whichever of them arrives last: every
// contributor stores its fp32 partial tile, then bumps the tile's arrival
// counter, and the one that completes the count adds the partials in k order
// (so the result does not depend on the arrival order), applies the
// epilogue and sets the counter back to zero. No workgroup waits for another.
struct GemmSched {
  int tiles_m, tiles_n, nk, group_n;
  int sk;         // 1: stream-K over gridDim.x workgroups
  int64_t total;  // tiles * nk
};

__device__ __forceinline__ void tile_coords(const GemmSched& s, int t, int& nt, int& mt) {
  const int per = s.group_n * s.tiles_m;
  const int gi = t / per, r = t - gi * per;
  const int first = gi * s.group_n;
  const int gsz = min(s.tiles_n - first, s.group_n);
  nt = first + r % gsz;
  mt = r / gsz;
}

// Stream-K: workgroup g owns iterations [floor(g T / G), floor((g+1) T / G)).
__device__ __forceinline__ int64_t sk_begin(int g, int64_t total, int G) {
  return (int64_t)g * total / G;
}
__device__ __forceinline__ int sk_owner(int64_t i, int64_t total, int G) {
  return (int)(((i + 1) * G - 1) / total);
}

// NS weight stages and NSX activation stages (NSX = NS, or one more or one
// fewer with two stages of the other): the loads of weight slab j + NS - 1
// and activation slab j + NSX - 1 are in flight while slab j is multiplied.
template <int BN, int BM, int NS, int SPR, bool SK, int EPI, int NW = 4, int NSX = NS>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4)))
void gemm_ring(GemmArgs a, GemmSched sc) {
  constexpr int BK = 64;
  using T = RTile<BN, BM, BK, NS, NW>;
  static_assert(NSX == NS || (NS == 2 && NSX == 3) || (NS == 3 && NSX == 2),
                "stage counts: equal, or 2 and 3");
  constexpr int CPR = T::CPR, RPI = T::RPI, WN = T::WN, WM = T::WM, TN = T::TN, TM = T::TM;
  constexpr int LPS = T::LPS;
  static_assert((EPI != EPI_SWIGLU && EPI != EPI_QKV_ROPE) || (WN % 32) == 0,
                "SwiGLU and RoPE need 32-row pairs");
  constexpr int X_BYTES = BM * BK * 2;
  __shared__ __attribute__((aligned(1024))) char smem[NS * T::W_BYTES + NSX * X_BYTES];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1;
  const int G = gridDim.x;
  int l = blockIdx.x;  // consecutive logical workgroups on one XCD
  if ((G & 7) == 0) l = (l & 7) * (G >> 3) + (l >> 3);

  const int kp = (a.K + 63) & ~63;
  const v4i_t rw = buf_rsrc(a.W, (uint64_t)a.N * kp * 2);
  const v4i_t rx = buf_rsrc(a.X, (uint64_t)a.M * a.ldx * 2);
  const int lrow = lane / CPR;
  const int lchunk = chunk_pos<CPR>(lrow, lane % CPR);  // row base is a multiple of RPI
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int vw = lane * 16;
  const int sw_slab = (a.N / 8) * 1024;
  const int sx_step = RPI * (int)a.ldx * 2;
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) char*)smem;
  // weight stages first, then the activation stages
  const uint32_t lds_w = lds0 + wave_u * (BN / NW) * BK * 2;
  const uint32_t lds_x = lds0 + NS * T::W_BYTES + wave_u * (BM / NW) * BK * 2;
  const int fr = lane & 15, g = lane >> 4;

  f32x4_v acc[TN][TM];

  // acc = sum over k steps [k0, k1) of tile (n0, m0)
  // QKV projection with RoPE, data-parallel tiles: the tile's token
  // positions and slots, and its cos/sin rows when they fit in registers, are
  // requested right after the main loop's first operand loads, so their round
  // trips overlap the pipeline start instead of delaying the epilogue. (Extra
  // loads only make the vmcnt waits of the ring stricter: loads complete in
  // order.)
  constexpr bool ROPE_PRE = EPI == EPI_QKV_ROPE && !SK;
  // (the cos/sin rows take 4 TN TM registers: with eight waves, two per
  // SIMD, only the small tiles have room; 256 x 256 spilled 100 registers)
  constexpr bool ROPE_TAB = ROPE_PRE && TN * TM <= (NW == 4 ? 32 : 16);
  constexpr int RJ = ROPE_PRE ? TM : 1, RJT = ROPE_TAB ? TM : 1, RI = ROPE_TAB ? TN / 2 : 1;
  int r_pos[RJ], r_slot[RJ];
  float4 r_cos[RJT][RI], r_sin[RJT][RI];
  auto rope_fetch = [&](int n0, int m0) {
    if constexpr (ROPE_PRE) {
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int m = m0 + wm * WM + j * 16 + fr;
        const bool in = m < a.M;
        r_pos[j] = in ? a.rope_pos[m] : 0;
        r_slot[j] = in ? a.rope_slot[m] : -1;
      }
      if constexpr (ROPE_TAB) {
        const int qk = a.rope_q_cols + a.rope_kv_cols;
#pragma unroll
        for (int j = 0; j < TM; ++j)
#pragma unroll
          for (int ip = 0; ip < TN / 2; ++ip) {
            const int n = n0 + wn * WN + ip * 32 + g * 4;
            const int64_t o = rope_tab_off(a, r_pos[j], n < qk ? n : 0);
            r_cos[j][ip] = *reinterpret_cast<const float4*>(a.rope_cos + o);
            r_sin[j][ip] = *reinterpret_cast<const float4*>(a.rope_sin + o);
          }
      }
    }
  };

  auto mainloop = [&](int n0, int m0, int k0, int k1, auto&& after_issue) {
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j) acc[i][j] = f32x4_v{0.f, 0.f, 0.f, 0.f};
    // weights: block (kt, n0/8 + wave * BN/(8 NW) + q) of the tiled format
    const int sw_base = (n0 / 8 + wave_u * (BN / NW / 8)) * 1024;
    const int vx = ((m0 + wave * (BM / NW) + lrow) * (int)a.ldx + lchunk * 8) * 2;
    // load q of a step (0 <= q < LPS): the operand whose slab is due sooner
    // goes first (weights when the look-aheads are equal)
    constexpr int AW = NS - 1, AX = NSX - 1;          // look-ahead in steps
    constexpr bool XFIRST = AX < AW;
    constexpr int FIRST = XFIRST ? T::XI : T::WI, SECOND = LPS - FIRST;
    auto issue_w = [&](int stage, int kt, int q) {
      dma16(rw, vw, sw_base + kt * sw_slab + q * 1024, lds_w + stage * T::W_BYTES + q * 1024);
    };
    auto issue_x = [&](int stage, int kt, int q) {
      dma16(rx, vx, q * sx_step + kt * BK * 2, lds_x + stage * X_BYTES + q * 1024);
    };
    // the loads of a step are spread over the first SPR/4 of the row-tile
    // steps of the current slab's multiplication
    constexpr int STEPS = TN * (BK / 32), USE = STEPS * SPR / 4;
    static_assert(USE >= 1, "spread");
    auto issue_part = [&](int j, int step, bool more_w, bool more_x) {
      if (step < USE) {
#pragma unroll
        for (int q = step * LPS / USE; q < (step + 1) * LPS / USE; ++q) {
          const bool first = q < FIRST;
          const bool is_x = first == XFIRST;
          const int qq = first ? q : q - FIRST;
          if (is_x) {
            if (more_x) issue_x((j + AX) % NSX, k0 + j + AX, qq);
          } else if (more_w) {
            issue_w((j + AW) % NS, k0 + j + AW, qq);
          }
        }
      }
    };
    // Step j issues the loads of weight slab j + AW and activation slab
    // j + AX while it multiplies slab j. The issue is behind a (uniform)
    // branch on purpose: it splits the step into scheduling regions, without
    // which the register allocator shuffles the accumulators between MFMAs.
    // Loads complete in issue order, so before slab j + 1 the wave waits
    // until only the loads issued after slab j + 1's last one are
    // outstanding: with equal look-aheads the (AW - 1) later steps' loads,
    // else the second operand's loads of step j.
    const int n = k1 - k0;
    // prologue: the loads of the virtual steps -max(AW, AX) .. -1, in the
    // same order as the steady state
#pragma unroll
    for (int v = -(AW > AX ? AW : AX); v < 0; ++v) {
      const int tw = v + AW, tx = v + AX;   // slabs this virtual step loads
      auto w_part = [&] {
        if (tw >= 0 && tw < n)
#pragma unroll
          for (int q = 0; q < T::WI; ++q) issue_w(tw % NS, k0 + tw, q);
      };
      auto x_part = [&] {
        if (tx >= 0 && tx < n)
#pragma unroll
          for (int q = 0; q < T::XI; ++q) issue_x(tx % NSX, k0 + tx, q);
      };
      if (XFIRST) { x_part(); w_part(); } else { w_part(); x_part(); }
    }
    after_issue();
    // before slab 0: what the prologue issued after slab 0's loads
    if constexpr (AW == AX) {
      if (n >= NS - 1) wait_vm<(NS - 2) * LPS>();
      else wait_vm<0>();
    } else {
      if (n >= 2) wait_vm<SECOND>();
      else wait_vm<0>();
    }
    wg_barrier();
    constexpr int PD = ring_pd<TN>();
    bf16x8_v fa[PD + 1], fb[2][TM];
    for (int j = 0; j < n; ++j) {
      const bool more_w = j + AW < n, more_x = j + AX < n;
      const bf16_t* sw = reinterpret_cast<const bf16_t*>(smem + (j % NS) * T::W_BYTES);
      const bf16_t* sx =
          reinterpret_cast<const bf16_t*>(smem + NS * T::W_BYTES + (j % NSX) * X_BYTES);
      ring_stage<BN, BM, BK, NS, NW, TN, TM, PD>(acc, fa, fb, sw, sx, wn, wm, fr, g, j > 0, [&](int step) {
        issue_part(j, step, more_w, more_x);
      });
      if constexpr (AW == AX) {
        if (more_w) wait_vm<(NS - 2) * LPS>();
        else wait_vm<0>();
      } else {
        if (more_w && more_x) wait_vm<SECOND>();
        else wait_vm<0>();
      }
      wg_barrier();
    }
    // the last stage's deferred row tile
#pragma unroll
    for (int jj = 0; jj < TM; ++jj)
      acc[TN - 1][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[(2 * TN - 1) % (PD + 1)], fb[1][jj], acc[TN - 1][jj], 0, 0, 0);
  };

  auto epilogue = [&](int n0, int m0) {
    const int fq = g * 4;
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int m = m0 + wm * WM + j * 16 + fr;
      if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int i = 0; i < TN; i += 2)
          store_swiglu(a, m, (n0 + wn * WN + i * 16) / 2 + fq, acc[i][j], acc[i + 1][j]);
      } else if constexpr (EPI == EPI_QKV_ROPE) {
        int pos, slot;
        if constexpr (ROPE_PRE) {
          pos = r_pos[j];
          slot = r_slot[j];
        } else {
          const bool in = m < a.M;
          pos = in ? a.rope_pos[m] : 0;
          slot = in ? a.rope_slot[m] : -1;
        }
        const int qk = a.rope_q_cols + a.rope_kv_cols;
#pragma unroll
        for (int i = 0; i < TN; i += 2) {
          const int n = n0 + wn * WN + i * 16 + fq;
          float4 cv, sv;
          if constexpr (ROPE_TAB) {
            cv = r_cos[j][i / 2];
            sv = r_sin[j][i / 2];
          } else {
            const int64_t o = rope_tab_off(a, pos, n < qk ? n : 0);
            cv = *reinterpret_cast<const float4*>(a.rope_cos + o);
            sv = *reinterpret_cast<const float4*>(a.rope_sin + o);
          }
          store_qkv_rope(a, m, slot, n, acc[i][j], acc[i + 1][j], cv, sv);
        }
      } else {
#pragma unroll
        for (int i = 0; i < TN; ++i) store4<EPI>(a, m, n0 + wn * WN + i * 16 + fq, acc[i][j]);
      }
    }
  };

  if constexpr (!SK) {
    int nt, mt;
    tile_coords(sc, l, nt, mt);
    mainloop(nt * BN, mt * BM, 0, sc.nk, [&] { rope_fetch(nt * BN, mt * BM); });
    epilogue(nt * BN, mt * BM);
  } else {

  // stream-K: partial tiles live at part[(2 * g + slot) * BN * BM], slot 0
  // for a workgroup's first segment and 1 for its last, in the lane order of
  // the accumulators (coalesced 1 KiB per fragment). They are written and
  // read with device-scope (sc1) accesses, which are coherent across the
  // XCDs' L2 caches on their own; a writer waits for its stores to complete
  // before its arrival is counted, so the last arrival sees every partial
  // without any cache-wide write-back or invalidation.
  constexpr int TILE_F = BN * BM;
  constexpr int kSc1 = 16;  // cache-policy bit: device scope
  typedef unsigned u32x4_v __attribute__((ext_vector_type(4)));
  const __amdgpu_buffer_rsrc_t rp =
      __builtin_amdgcn_make_buffer_rsrc(a.part, 0, 0x7FFFFFFF, kRsrcWord3);
  auto frag_off = [&](int i, int j) { return (((i * TM + j) * NW + wave) * 64 + lane) * 16; };
  const int64_t beg = sk_begin(l, sc.total, G), end = sk_begin(l + 1, sc.total, G);
  for (int64_t it = beg; it < end;) {
    const int t = (int)(it / sc.nk);
    const int k0 = (int)(it - (int64_t)t * sc.nk);
    const int k1 = (int)min<int64_t>(sc.nk, k0 + (end - it));
    int nt, mt;
    tile_coords(sc, t, nt, mt);
    mainloop(nt * BN, mt * BM, k0, k1, [] {});
    if (k0 > 0 || k1 < sc.nk) {
      const int slot = it == beg ? 0 : 1;
      const int mine = (2 * l + slot) * TILE_F * 4;
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_v, acc[i][j]), rp,
                                                 frag_off(i, j), mine, kSc1);
      const int g0 = sk_owner((int64_t)t * sc.nk, sc.total, G);
      const int g1 = sk_owner((int64_t)(t + 1) * sc.nk - 1, sc.total, G);
      wait_vm<0>();
      __syncthreads();
      if (tid == 0) {
        const uint32_t prev =
            __hip_atomic_fetch_add(a.flags + t, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_last = prev == (uint32_t)(g1 - g0);
      }
      __syncthreads();
      if (s_last) {
        // running sum over contributors in k order; the partials before this
        // workgroup's own go into `pre`, the rest straight into acc (16
        // fragments per batch of loads, 8 or 16)
        constexpr int FR = TN * TM, HB = FR > 16 ? 8 : FR;
#pragma unroll
        for (int f0 = 0; f0 < FR; f0 += HB) {
          f32x4_v pre[HB];
          bool after = false;
          for (int c = g0; c <= g1; ++c) {
            if (c == l) {
              if (c != g0) {
#pragma unroll
                for (int u = 0; u < HB; ++u)
                  acc[(f0 + u) / TM][(f0 + u) % TM] = pre[u] + acc[(f0 + u) / TM][(f0 + u) % TM];
              }
              after = true;
              continue;
            }
            const int cs = sk_begin(c, sc.total, G) / sc.nk == t ? 0 : 1;
            f32x4_v v[HB];
#pragma unroll
            for (int u = 0; u < HB; ++u)
              v[u] = __builtin_bit_cast(
                  f32x4_v, __builtin_amdgcn_raw_buffer_load_b128(
                               rp, frag_off((f0 + u) / TM, (f0 + u) % TM),
                               __builtin_amdgcn_readfirstlane((2 * c + cs) * TILE_F * 4), kSc1));
            if (after) {
#pragma unroll
              for (int u = 0; u < HB; ++u) acc[(f0 + u) / TM][(f0 + u) % TM] += v[u];
            } else if (c == g0) {
#pragma unroll
              for (int u = 0; u < HB; ++u) pre[u] = v[u];
            } else {
#pragma unroll
              for (int u = 0; u < HB; ++u) pre[u] += v[u];
            }
          }
        }
        if (tid == 0) __hip_atomic_store(a.flags + t, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        epilogue(nt * BN, mt * BM);
      }
    } else {
      epilogue(nt * BN, mt * BM);
    }
    it += k1 - k0;
  }
  }
}

// ------------------------------------------------------------ skinny (decode)
//
// A workgroup owns 16 * NF weight rows and all M <= 64 tokens; its WV waves
// split the 64-column slabs of K. For one slab, the 2 NF row blocks of the
// workgroup are adjacent 1 KiB blocks. Each is read by one wave-wide 16-byte
// load with lane L taking bytes [16 L, 16 L + 16) (a whole block per
// instruction, non-temporal: the weights are streamed once per call), then
// stored unchanged into the wave's own LDS buffer and read back in the MFMA
// fragment order: lane (row fr, group g) takes chunk 4 ks + g of its row for
// the ks-th 32-k MFMA. The buffer keeps the block's XOR-swizzled chunk order,
// so the fragment reads are free of bank conflicts. (Loading the fragments
// straight from global memory makes every instruction touch half of each of
// 16 rows; the whole-block loads stream 10-30% faster on MI355X.) The loads
// of the next slab group are issued before the current one is multiplied.
//
// The activations (the B operand, tokens on the MFMA columns) are loaded in
// fragment order, lane (fr, g) taking chunk 4 ks + g of token fr: 64 bytes of
// each of 16 rows per instruction. With XS they take the weights' route
// instead: instruction h of a 16-token chunk reads whole 128-byte rows of
// tokens 8h .. 8h + 7 (lane L: token 8h + L/8, chunk (L % 8) ^ (L / 8)) and
// stores them to position 64 h + L of the wave's activation buffer, which
// then has the layout of a weight tile's image and is read like one. The
// MFMA operands are the same either way; staging pays off once many tokens
// share the call (8B-shape o and down projections at 16 tokens, MI355X:
// 12.3 -> 9.7 and 26.5 -> 23.5 us) and costs about 0.5 us at one token.

// With NORM, X is the un-normalised residual stream and the GEMM applies the
// RMSNorm of its rows itself: each loaded activation chunk is multiplied by
// the norm gain (and rounded to bf16 like a stored activation), the squares
// of the raw values are summed along the way, and the epilogue scales each
// token's outputs by 1 / sqrt(mean square + eps). Used for decode, where the
// separate norm kernel would cost a launch per projection.
template <int NF, int MCH, int U, int EPI, bool NORM, int WV, bool XS>
__global__ __launch_bounds__(64 * WV) void gemm_skinny(GemmArgs a) {
  static_assert(EPI != EPI_SWIGLU || (NF % 2) == 0, "SwiGLU needs gate/up tile pairs");
  // the norm's sums of squares follow the fragment-order loads; keeping one
  // order for every batch size keeps a token's result independent of M
  static_assert(!(NORM && XS), "staged activations are built without the fused norm");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16 * NF;
  const int kp = (a.K + 63) & ~63;
  const int nslab = kp / 64;
  const int sq = (nslab + WV - 1) / WV;  // slabs per wave
  const int sb = wave * sq, se = min(nslab, sb + sq);
  const int fr = lane & 15, g = lane >> 4;
  const int64_t slab_bytes = (int64_t)(a.N / 8) * 1024;
  // instruction (f, h) of a slab reads row block n0 / 8 + 2 f + h (N % 16 == 0,
  // so a 16-row tile is either wholly inside the matrix or wholly outside)
  const char* wbase = reinterpret_cast<const char*>(a.W) + (int64_t)(n0 / 8) * 1024 + lane * 16;
  bool wok[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) wok[f] = n0 + 16 * f < a.N;
  const int r8 = fr % 8;
  // 16-byte position of lane (fr, g)'s row inside the 2 KiB image of a 16-row tile
  const int fpos = (fr / 8) * 64 + r8 * 8;
  // activation rows. XS: load i = 2 c + h (instruction h of token chunk c)
  // reads token 8 i + L / 8, at 16-byte chunk (L % 8) ^ (L / 8) of each slab;
  // otherwise load c reads token 16 c + fr (its chunk offset added per load)
  constexpr int XH = XS ? 2 : 1;
  const int xr = lane >> 3, xc = (lane & 7) ^ (lane >> 3);
  const bf16_t* xrow[MCH * XH];
#pragma unroll
  for (int i = 0; i < MCH * XH; ++i) {
    const int m = XS ? 8 * i + xr : 16 * i + fr;
    xrow[i] = (m < a.M) ? a.X + (int64_t)m * a.ldx + (XS ? xc * 8 : 0) : nullptr;
  }
  // per wave and slab: the weight tiles' images, then with XS the activation
  // chunks' images (16-byte units)
  __shared__ pack8 wlds[WV][U][(NF + (XS ? MCH : 0)) * 128];

  f32x4_v acc[NF][MCH];
  float ssq[MCH];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int c = 0; c < MCH; ++c) acc[f][c] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < MCH; ++c) ssq[c] = 0.f;

  pack8 wv[U][NF][2];
  auto load_w = [&](int s0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sl = s0 + u;
      const bool ok = sl < se;
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int h = 0; h < 2; ++h)
          wv[u][f][h] = (ok && wok[f]) ? ld16_nt(wbase + sl * slab_bytes + (2 * f + h) * 1024)
                                       : zero8();
    }
  };
  if (sb < se) load_w(sb);
  for (int s0 = sb; s0 < se; s0 += U) {
    // this wave's buffer: the previous group's fragment reads were issued
    // before these stores, and one wave's LDS operations run in order
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int h = 0; h < 2; ++h) wlds[wave][u][(2 * f + h) * 64 + lane] = wv[u][f][h];
    if (s0 + U < se) load_w(s0 + U);
    // activations: XS, whole rows (stored below); else fragment order, xv[c][u][ks]
    pack8 xv[MCH][U][2], gv[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sl = s0 + u;
      const bool ok = sl < se;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int chunk = ks * 4 + g;
#pragma unroll
        for (int c = 0; c < MCH; ++c) {
          if constexpr (XS)
            xv[c][u][ks] = (ok && xrow[2 * c + ks]) ? ld16(xrow[2 * c + ks] + sl * 64) : zero8();
          else
            xv[c][u][ks] = (ok && xrow[c]) ? ld16(xrow[c] + sl * 64 + chunk * 8) : zero8();
        }
        if constexpr (NORM) gv[u][ks] = ok ? ld16(a.norm_gain + sl * 64 + chunk * 8) : zero8();
      }
    }
    if constexpr (NORM) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int c = 0; c < MCH; ++c) {
            pack8& x = xv[c][u][ks];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float x0 = lo_bf(x.w[e]), x1 = hi_bf(x.w[e]);
              ssq[c] += x0 * x0 + x1 * x1;
              x.w[e] = pack2bf(x0 * lo_bf(gv[u][ks].w[e]), x1 * hi_bf(gv[u][ks].w[e]));
            }
          }
    }
    if constexpr (XS) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int c = 0; c < MCH; ++c)
#pragma unroll
          for (int h = 0; h < 2; ++h) wlds[wave][u][NF * 128 + (2 * c + h) * 64 + lane] = xv[c][u][h];
    }
    asm volatile("" ::: "memory");  // keep the fragment reads after the stores
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        if constexpr (XS) {  // the fragments from the staged image (read like a weight tile's)
#pragma unroll
          for (int c = 0; c < MCH; ++c)
            xv[c][u][ks] = wlds[wave][u][(NF + c) * 128 + fpos + ((ks * 4 + g) ^ r8)];
        }
#pragma unroll
        for (int f = 0; f < NF; ++f) {
          const pack8 w = wlds[wave][u][f * 128 + fpos + ((ks * 4 + g) ^ r8)];
#pragma unroll
          for (int c = 0; c < MCH; ++c)
            acc[f][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                as_bf16x8(w), as_bf16x8(xv[c][u][ks]), acc[f][c], 0, 0, 0);
        }
      }
    asm volatile("" ::: "memory");  // and the next stores after these reads
  }

  __shared__ f32x4_v red[WV - 1][NF][MCH][64];
  __shared__ float red_ss[WV][MCH][16];
  if constexpr (NORM) {
    // the 4 k-groups of a token (lanes fr, fr+16, fr+32, fr+48), then waves
#pragma unroll
    for (int c = 0; c < MCH; ++c) {
      ssq[c] += __shfl_xor(ssq[c], 16, 64);
      ssq[c] += __shfl_xor(ssq[c], 32, 64);
      if (g == 0) red_ss[wave][c][fr] = ssq[c];
    }
  }
  if (wave > 0) {
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int c = 0; c < MCH; ++c) red[wave - 1][f][c][lane] = acc[f][c];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < WV - 1; ++w)
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int c = 0; c < MCH; ++c) acc[f][c] += red[w][f][c][lane];
  if constexpr (NORM) {
#pragma unroll
    for (int c = 0; c < MCH; ++c) {
      float tot = red_ss[0][c][fr];
#pragma unroll
      for (int w = 1; w < WV; ++w) tot += red_ss[w][c][fr];
      const float inv = 1.0f / sqrtf(tot / (float)a.K + a.norm_eps);
#pragma unroll
      for (int f = 0; f < NF; ++f) acc[f][c] *= inv;
    }
  }

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

template <int NF, int MCH, int U, int WV, bool XS, bool NORM>
hipError_t dispatch_skinny_norm(const GemmArgs& a, int epi, hipStream_t s) {
  const int grid = (a.N + 16 * NF - 1) / (16 * NF);
  const dim3 blk(64 * WV);
  switch (epi) {
    case EPI_STORE:
      hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_STORE, NORM, WV, XS>), dim3(grid), blk, 0, s, a);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_RESID, NORM, WV, XS>), dim3(grid), blk, 0, s, a);
      break;
    case EPI_SWIGLU:
      if constexpr (NF % 2 == 0) {
        hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_SWIGLU, NORM, WV, XS>), dim3(grid), blk, 0, s, a);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case EPI_F32:
      hipLaunchKernelGGL((gemm_skinny<NF, MCH, U, EPI_F32, NORM, WV, XS>), dim3(grid), blk, 0, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int NF, int MCH, int U, int WV, bool XS = false>
hipError_t dispatch_epi_skinny(const GemmArgs& a, int epi, hipStream_t s) {
  if (a.norm_gain) {
    // the fused norm is only built for one 16-token chunk (decode batches)
    if constexpr (MCH == 1 && !XS) return dispatch_skinny_norm<NF, 1, U, WV, false, true>(a, epi, s);
    else return hipErrorInvalidValue;
  }
  return dispatch_skinny_norm<NF, MCH, U, WV, XS, false>(a, epi, s);
}

// The skinny variants built for one 16-token chunk, as (rows per workgroup /
// 16, slabs unrolled per wave, waves per workgroup, staged activations): the
// ones the selection in gemm() takes.
#define HS_SKINNY_MCH1(X)                                                                      \
  X(1, 1, 8, false) X(2, 1, 8, false) X(2, 1, 4, false) X(4, 1, 4, false) X(2, 1, 2, false) \
  X(4, 1, 2, false) X(8, 1, 2, false) X(1, 1, 16, false) X(3, 1, 16, false) X(1, 1, 16, true)

hipError_t dispatch_skinny1(const GemmArgs& a, int epi, int nf, int u, int wv, bool xs,
                            hipStream_t s) {
#define HS_SKINNY_CASE(NF_, U_, WV_, XS_)                  \
  if (nf == NF_ && u == U_ && wv == WV_ && xs == XS_) \
    return dispatch_epi_skinny<NF_, 1, U_, WV_, XS_>(a, epi, s);
  HS_SKINNY_MCH1(HS_SKINNY_CASE)
#undef HS_SKINNY_CASE
  return hipErrorInvalidValue;
}

template <int BN, int BM, int NS, int SPR, bool SK, int NW = 4, int NSX = NS>
hipError_t dispatch_ring(const GemmArgs& a, int epi, const GemmSched& sc, int grid, hipStream_t s) {
  const dim3 blk(64 * NW);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_ring<BN, BM, NS, SPR, SK, EPI_STORE, NW, NSX>), dim3(grid), blk, 0, s, a, sc); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_ring<BN, BM, NS, SPR, SK, EPI_RESID, NW, NSX>), dim3(grid), blk, 0, s, a, sc); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_ring<BN, BM, NS, SPR, SK, EPI_SWIGLU, NW, NSX>), dim3(grid), blk, 0, s, a, sc); break;
    case EPI_F32: hipLaunchKernelGGL((gemm_ring<BN, BM, NS, SPR, SK, EPI_F32, NW, NSX>), dim3(grid), blk, 0, s, a, sc); break;
    case EPI_QKV_ROPE: hipLaunchKernelGGL((gemm_ring<BN, BM, NS, SPR, SK, EPI_QKV_ROPE, NW, NSX>), dim3(grid), blk, 0, s, a, sc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

struct RingCfg {
  const char* name;
  int bn, bm;
  bool sk_ok;  // has a stream-K build
};
const RingCfg kRing[] = {{"256x256", 256, 256, false}, {"256x128", 256, 128, true},
                         {"128x128", 128, 128, true},  {"192x256", 192, 256, false},
                         {"192x128", 192, 128, false}};

// 256 x 256: 2 stages (128 KiB of LDS); 192 x 256: 3 weight stages and 2
// activation stages (136 KiB); the next slabs' loads issued in the first
// half of the current one's multiplication. 256 x 128: 3 stages, loads
// spread over the whole step. 192 x 128 (160 KiB) and 128 x 128: 4 stages.
hipError_t launch_ring(const RingCfg& c, const GemmArgs& a, int epi, const GemmSched& sc,
                       int grid, hipStream_t s) {
  // Eight waves (two per SIMD: one wave's LDS reads and barrier waits hide
  // behind the other's MFMAs) unless HS_GEMM_WAVES=4 (tuning only). The
  // 512-token 7B stage, MI355X: o 36.5 -> 32.9 us, down 69.8 -> 65.5, QKV
  // 66.7 -> 59.7, gate/up unchanged; 8192 tokens: o 240 -> 219, QKV 674 -> 647.
  // Each output is still summed by one wave in k order, so the bits do not
  // change.
  static const char* waves = getenv("HS_GEMM_WAVES");
  const bool w4 = waves && atoi(waves) == 4;
  if (c.bn == 256 && c.bm == 256)
    return w4 ? dispatch_ring<256, 256, 2, 2, false>(a, epi, sc, grid, s)
              : dispatch_ring<256, 256, 2, 2, false, 8>(a, epi, sc, grid, s);
  // 192 x 256: three weight stages and two activation stages (136 KiB),
  // the weights requested two slabs ahead. At a 512-token prompt every CU
  // runs one tile and each 64-k slab takes about 1.3 us, shorter than a
  // load's latency under load: 7B gate/up 91.0 -> 82.0 us (two of each:
  // 112 KiB; weights two ahead and activations one gave the same gain as
  // the reverse, and three of each does not fit). At 8192 tokens the
  // 256 x 256 tiles' longer slabs hide the latency: a third weight stage
  // there moved nothing beyond noise.
  if (c.bn == 192 && c.bm == 256)
    return w4 ? dispatch_ring<192, 256, 2, 2, false>(a, epi, sc, grid, s)
              : dispatch_ring<192, 256, 3, 2, false, 8, 2>(a, epi, sc, grid, s);
  if (c.bn == 192 && c.bm == 128)
    return w4 ? dispatch_ring<192, 128, 4, 4, false>(a, epi, sc, grid, s)
              : dispatch_ring<192, 128, 4, 4, false, 8>(a, epi, sc, grid, s);
  if (c.bn == 256 && c.bm == 128) {
    // stream-K 256 x 128 keeps four waves (its partial-tile reduction does
    // not fit the registers of eight: 125-138 spilled)
    if (sc.sk) return dispatch_ring<256, 128, 3, 4, true>(a, epi, sc, grid, s);
    return w4 ? dispatch_ring<256, 128, 3, 4, false>(a, epi, sc, grid, s)
              : dispatch_ring<256, 128, 3, 4, false, 8>(a, epi, sc, grid, s);
  }
  if (w4)
    return sc.sk ? dispatch_ring<128, 128, 4, 4, true>(a, epi, sc, grid, s)
                 : dispatch_ring<128, 128, 4, 4, false>(a, epi, sc, grid, s);
  return sc.sk ? dispatch_ring<128, 128, 4, 4, true, 8>(a, epi, sc, grid, s)
               : dispatch_ring<128, 128, 4, 4, false, 8>(a, epi, sc, grid, s);
}

int device_cus() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cus[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

const char* kEpiName[5] = {"store", "resid", "swiglu", "f32", "qkv_rope"};

}  // namespace

hipError_t gemm(const GemmArgs& a, int epi, hipStream_t s, LaunchInfo* info) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return hipErrorInvalidValue;
  if (epi < 0 || epi > 4) return hipErrorInvalidValue;
  // head-interleaved q/k rows: whole heads of 64 or 128, then as many v columns as k
  if (a.rope_q_cols || a.rope_kv_cols) {
    const int d = a.rope_d;
    if ((d != 64 && d != 128) || a.rope_q_cols <= 0 || a.rope_kv_cols <= 0 ||
        (a.rope_q_cols % d) || (a.rope_kv_cols % d) || a.rope_q_cols + 2 * a.rope_kv_cols != a.N)
      return hipErrorInvalidValue;
  }
  if (epi == EPI_QKV_ROPE &&
      (!a.rope_q_cols || !a.rope_pos || !a.rope_slot || !a.rope_cos || !a.rope_sin ||
       !a.rope_pool || a.rope_max_pos <= 0 || (a.ldy % 8) ||
       ((uintptr_t)a.rope_cos & 15) || ((uintptr_t)a.rope_sin & 15) ||
       ((uintptr_t)a.rope_pool & 15)))
    return hipErrorInvalidValue;
  const int64_t kp = (a.K + 63) / 64 * 64;
  if ((a.K % 8) || (a.N % 16) || (a.ldx % 8) || (a.ldy % 4)) return hipErrorInvalidValue;
  if ((a.K % 64) && a.ldx < kp) return hipErrorInvalidValue;
  if (epi == EPI_SWIGLU && (a.N % 32)) return hipErrorInvalidValue;
  if (epi == EPI_RESID && (!a.R || (a.ldr % 4))) return hipErrorInvalidValue;
  if (((uintptr_t)a.X | (uintptr_t)a.W | (uintptr_t)a.Y) & 15) return hipErrorInvalidValue;
  if (a.norm_gain && (a.M > 16 || (a.K % 64) || ((uintptr_t)a.norm_gain & 15)))
    return hipErrorInvalidValue;
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
    // a QKV projection with RoPE runs as a plain (head-order) store followed
    // by the rotation pass
    const int pe = epi == EPI_QKV_ROPE ? EPI_STORE : epi;
    const int mch = (a.M + 15) / 16;
    // Rows per workgroup (16 NF), 64-k slabs per load group (U), waves per
    // workgroup (WV) and staged activations (XS) for one token chunk, from
    // sweeps on MI355X over the decode projections of 7B, 8B and 13B models
    // at 1, 4, 8 and 16 tokens: o and down projections up to one row tile
    // per CU run sixteen waves of one row tile (7B down at 1 and 8 tokens:
    // 17.4 -> 16.2 and 18.2 -> 16.9 us against eight waves and two slabs per
    // group), with the activations staged from 8 tokens on; wider ones eight
    // waves, two row tiles above 4 tokens. QKV up to 8192 wide takes eight
    // waves, wide QKV and gate/up four; gate/up takes four row tiles per
    // workgroup once that still gives 1.5 workgroups per CU (8B, 13B: 38 and
    // 45 instead of 43 and 52 us); the LM head runs two waves over as many
    // row tiles as keep about a thousand workgroups (128256 wide: 155 instead
    // of 162-169 us). WV depends on the shape only, never on M, so that a
    // token's result (its k order) does not depend on how many tokens share
    // the call; XS changes only how the same operands reach the MFMAs.
    // HS_SKINNY_CFG="<NF>,<U>,<WV>[,<XS>]" forces a choice (tuning only; read
    // on every call so that a sweep can change it between calls).
    const char* force = getenv("HS_SKINNY_CFG");
    const int cus = device_cus();
    int nf = 1, u = 1, wv = 4, xs = 0;
    if (pe == EPI_F32) {
      nf = 2, wv = 2;
      while (nf < 8 && a.N / (16 * nf) > 1100) nf *= 2;
    } else if (pe == EPI_SWIGLU) {
      nf = (a.N / 64 >= cus + cus / 2) ? 4 : 2;
    } else if (pe == EPI_RESID) {
      wv = 8;
      if (a.N / 16 > cus) {
        nf = a.M > 4 ? 2 : 1;
      } else {
        wv = 16;
        xs = a.M >= 8;
      }
    } else if (pe == EPI_STORE) {
      nf = 2, wv = a.N <= 8192 ? 8 : 4;
      // three row tiles when that gives one workgroup per CU (7B QKV: 256 x
      // 48 rows; 21.5 -> 19.5 us)
      if (a.N % 48 == 0 && a.N / 48 <= cus && a.N / 48 > cus * 3 / 4) nf = 3, wv = 16;
    }
    if (force && *force) sscanf(force, "%d,%d,%d,%d", &nf, &u, &wv, &xs);
    if (pe == EPI_SWIGLU && (nf % 2)) nf = 2;
    if (mch == 1) {
      e = dispatch_skinny1(a, pe, nf, u, wv, xs != 0, s);
    } else if (pe == EPI_SWIGLU) {
      switch (mch) {
        case 2: e = dispatch_epi_skinny<2, 2, 2, 4>(a, pe, s); break;
        case 3: e = dispatch_epi_skinny<2, 3, 1, 4>(a, pe, s); break;
        default: e = dispatch_epi_skinny<2, 4, 1, 4>(a, pe, s); break;
      }
    } else {
      switch (mch) {
        case 2: e = dispatch_epi_skinny<1, 2, 2, 4>(a, pe, s); break;
        case 3: e = dispatch_epi_skinny<1, 3, 2, 4>(a, pe, s); break;
        default: e = dispatch_epi_skinny<1, 4, 1, 4>(a, pe, s); break;
      }
    }
    if (e == hipSuccess && epi == EPI_QKV_ROPE) {
      RopeKvArgs r{static_cast<bf16_t*>(a.Y), a.ldy, a.rope_pos, a.rope_slot, a.rope_cos,
                   a.rope_sin, a.rope_pool, a.M, a.rope_q_cols / a.rope_d,
                   a.rope_kv_cols / a.rope_d, a.rope_d, a.rope_max_pos};
      e = rope_kv(r, s, nullptr);
    }
    snprintf(name, sizeof name, "gemm_skinny_%s%s", a.norm_gain ? "norm_" : "", kEpiName[epi]);
  } else {
    // Configuration by a small cost model: a data-parallel launch takes
    // rounds x (tile flops / per-CU rate of its tile shape); a stream-K launch
    // takes (flops / CUs) / its rate plus a fixed cost for the pipeline
    // start-ups and the partial-tile reductions. The rates are per-CU
    // TFLOP/s measured on MI355X with weights streamed from HBM.
    // HS_GEMM_CFG="<tile>[,dp|,sk][,g<n>]" forces a choice (tuning only; read
    // on every call so that a sweep can change it between calls).
    const int cus = device_cus();
    const int nk = (int)(kp / 64);
    struct Cand { const RingCfg* c; bool sk; double rate; };
    auto tiles_of = [&](const RingCfg& c) {
      return (long)((a.N + c.bn - 1) / c.bn) * ((a.M + c.bm - 1) / c.bm);
    };
    auto sk_room = [&](const RingCfg& c, long tiles) {
      const long g = std::min<long>(cus, tiles * nk / 4);
      return c.sk_ok && g >= 1 && a.part && a.flags && tiles <= a.flags_n &&
             2 * g * (int64_t)c.bn * c.bm <= a.part_floats;
    };
    // The 192-wide tiles cover more CUs when one round of tiles fills the
    // chip (512-token 7B prompt, MI355X: gate/up 230 tiles of 192 x 256
    // instead of 172 of 256 x 256, 102 instead of 118 us; QKV 256 tiles of
    // 192 x 128 instead of 192 of 256 x 128, 54 instead of 67 us); over
    // several rounds they lose to the 256-wide ones (4096-wide projections of
    // 8192 tokens: 20% slower), so they only run as a single round.
    const Cand cands[] = {{&kRing[0], false, 4.8}, {&kRing[1], false, 4.05},
                          {&kRing[2], false, 3.05}, {&kRing[2], true, 3.0},
                          {&kRing[3], false, 4.45}, {&kRing[4], false, 3.9}};
    const double sk_fixed_us = 10.0;
    const RingCfg* cfg = nullptr;
    bool sk = false;
    double best = 1e300;
    for (int i = 0; i < (int)(sizeof cands / sizeof cands[0]); ++i) {
      const RingCfg& c = *cands[i].c;
      const long tiles = tiles_of(c);
      double us;
      if (!cands[i].sk) {
        if (c.bn == 192 && tiles > cus) continue;
        const long rounds = (tiles + cus - 1) / cus;
        us = rounds * (2.0 * kp * c.bn * c.bm) / (cands[i].rate * 1e6);
      } else {
        if (!sk_room(c, tiles)) continue;
        us = (2.0 * a.M * (double)a.N * kp / cus) / (cands[i].rate * 1e6) + sk_fixed_us;
      }
      if (us < best) {
        best = us;
        cfg = &c;
        sk = cands[i].sk;
      }
    }
    int group = 8;
    const char* force = getenv("HS_GEMM_CFG");  // read per call (tuning sweeps)
    if (force && *force) {
      std::string f(force);
      for (const RingCfg& c : kRing)  // longest matching name wins
        if (f.compare(0, strlen(c.name), c.name) == 0 &&
            (f.size() == strlen(c.name) || f[strlen(c.name)] == ','))
          cfg = &c;
      if (f.find(",dp") != std::string::npos) sk = false;
      if (f.find(",sk") != std::string::npos) sk = true;
      const size_t gp = f.find(",g");
      if (gp != std::string::npos) group = std::max(1, atoi(f.c_str() + gp + 2));
    }
    GemmSched sc;
    sc.tiles_n = (a.N + cfg->bn - 1) / cfg->bn;
    sc.tiles_m = (a.M + cfg->bm - 1) / cfg->bm;
    sc.nk = nk;
    sc.group_n = group;
    const long tiles = (long)sc.tiles_n * sc.tiles_m;
    sc.total = (int64_t)tiles * nk;
    if (sk && !sk_room(*cfg, tiles)) sk = false;
    sc.sk = sk ? 1 : 0;
    const long grid = sk ? std::min<long>(cus, sc.total / 4) : tiles;
    if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
    e = launch_ring(*cfg, a, epi, sc, (int)grid, s);
    snprintf(name, sizeof name, "gemm_r%s%s_%s", cfg->name, sk ? "sk" : "", kEpiName[epi]);
  }
  if (info) {
    info->name = name;
    info->flops = flops;
    info->bytes = bytes;
  }
  return e;
}

}  // namespace hs
