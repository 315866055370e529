// Causal attention for prefill (flash-style, MFMA) and split-K paged decode.
//
// Prefill reads post-RoPE q, k and v straight from the QKV GEMM output (the
// whole prompt is in the call), one workgroup per (64-query tile, head).
// Decode reads the paged KV pools through each sequence's block table; the
// context is cut into fixed 128-token splits, so the split count depends on
// the context length only and the result is deterministic.
#include "hs_device.h"
#include "hs_kernels.h"

#include <stdlib.h>
#include <string.h>

#include <algorithm>

namespace hs {

// ------------------------------------------------------------------ prefill
//
// Wave w of the workgroup owns queries q0 + 16w .. q0 + 16w + 15. Scores are
// computed transposed, S^T[key][query] = K Q^T, so that each lane holds 16
// scores of ONE query (4 per 16-key subtile); the softmax statistics of a
// query then live in the 4 lanes l, l+16, l+32, l+48. P^T feeds the second
// MFMA as its B operand with the key order of each 32-key step permuted
// (lane group g, element e -> key 4g+e for e<4, 16+4g+e-4 otherwise). K and
// V are both staged row-major ([key][d]); the V^T fragments of the second
// MFMA come from transposing LDS reads (ds_read_b64_tr_b16: within each
// 16-lane group, lane o receives element o % 4 of the 4-element rows
// addressed by lanes o / 4, o / 4 + 4, o / 4 + 8 and o / 4 + 12), two per
// fragment, whose row addresses follow the same key permutation.

typedef short s16x4_v __attribute__((ext_vector_type(4)));

// KS = 2 (key split, 8 waves on a 64-query tile): waves w and w + 4 own the
// same 16 queries; the first takes the even key blocks, the second the odd
// ones, each half of the workgroup staging its own block, and at the end the
// second hands its running max, sum and output to the first through LDS
// (a fixed merge order). Two waves per SIMD hide each block's serial chain
// (score MFMAs, cross-lane max, exp2, P V MFMAs) when the tiles fill at most
// one workgroup per CU.
template <int D, int NW, int KS>
__global__ __launch_bounds__(64 * NW * KS) void attn_prefill_kernel(AttnPrefillArgs a, float scale_log2) {
  static_assert(KS == 1 || (KS == 2 && NW == 4), "key split: 2 x 4 waves");
  constexpr int NT = 64 * NW;   // threads staging one key block
  constexpr int QT = 16 * NW;   // queries per workgroup
  constexpr int KB = 64;        // keys per block
  constexpr int LK = D + 8;     // padded K row in LDS
  constexpr int LV = D + 16;     // padded V row in LDS: the 8-byte rows of a transposing
                                // read (4 keys x 4 column quads per 16 lanes) on distinct banks
  constexpr int CPK = D / 8;    // 16-byte chunks per key row
  constexpr int KPP = NT / CPK; // key rows per load pass
  constexpr int PASS = KB / KPP;
  static_assert(KB % KPP == 0 && (KPP % 2) == 0, "load mapping");
  __shared__ __attribute__((aligned(16))) bf16_t sKb[KS][KB * LK];
  __shared__ __attribute__((aligned(16))) bf16_t sVb[KS][KB * LV];

  const int part = KS == 1 ? 0 : threadIdx.x / NT;  // key parity of this half
  bf16_t* const sK = sKb[part];
  bf16_t* const sV = sVb[part];
  const int tid = threadIdx.x % NT, lane = tid & 63, wave = tid >> 6;
  // Workgroup b runs on XCD b mod 8: the logical (tile, head) order puts the
  // tiles of one head, which read the same keys and values, on one XCD (and
  // its L2) instead of spreading them over all eight.
  const int nwg = gridDim.x * gridDim.y;
  int lwg = blockIdx.x + blockIdx.y * gridDim.x;
  if ((nwg & 7) == 0) lwg = (lwg & 7) * (nwg >> 3) + (lwg >> 3);
  const int tile = lwg % gridDim.x;
  const int seq = a.tiles[2 * tile], q0 = a.tiles[2 * tile + 1];
  const int h = lwg / gridDim.x;
  const int kh = h / (a.n_heads / a.n_kv_heads);
  const int base = a.cu[seq], len = a.cu[seq + 1] - base;
  const int fr = lane & 15, g = lane >> 4;

  const int qw0 = q0 + wave * 16;        // first query of this wave
  const int qrow = qw0 + fr;             // this lane's query (position in sequence)
  bf16x8_v qf[D / 32];
#pragma unroll
  for (int ks = 0; ks < D / 32; ++ks) {
    pack8 v = zero8();
    if (qrow < len) v = ld16(a.qkv + (int64_t)(base + qrow) * a.ld + h * D + ks * 32 + g * 8);
    qf[ks] = as_bf16x8(v);
  }

  f32x4_v o[D / 16];
#pragma unroll
  for (int i = 0; i < D / 16; ++i) o[i] = f32x4_v{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int kend = min(len, q0 + QT);
  const int n_kb = (kend + KB - 1) / KB;
  const bf16_t* kbase = a.qkv + (int64_t)base * a.ld + (a.n_heads + kh) * D;
  const bf16_t* vbase = a.qkv + (int64_t)base * a.ld + (a.n_heads + a.n_kv_heads + kh) * D;
  const int lkey = tid / CPK, lcol = (tid % CPK) * 8;  // this thread's key row / column

  pack8 kreg[PASS], vreg[PASS];
  auto fetch = [&](int kb) {
#pragma unroll
    for (int p = 0; p < PASS; ++p) {
      const int key = kb * KB + p * KPP + lkey;
      kreg[p] = key < len ? ld16(kbase + (int64_t)key * a.ld + lcol) : zero8();
      vreg[p] = key < len ? ld16(vbase + (int64_t)key * a.ld + lcol) : zero8();
    }
  };
  fetch(part);  // past the last block: zero rows, never multiplied

  for (int kb0 = 0; kb0 < n_kb; kb0 += KS) {
    const int kb = kb0 + part;
    const int k0 = kb * KB;
    __syncthreads();  // every wave is done with the previous block
#pragma unroll
    for (int p = 0; p < PASS; ++p) {
      const int key = p * KPP + lkey;
      st16(&sK[key * LK + lcol], kreg[p]);
      st16(&sV[key * LV + lcol], vreg[p]);
    }
    __syncthreads();
    if (kb0 + KS < n_kb) fetch(kb + KS);  // in flight during this block's MFMAs
    if (kb >= n_kb || k0 > qw0 + 15) continue;  // no such block, or in this wave's future

    f32x4_v s[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      s[t] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / 32; ++ks) {
        const bf16x8_v kf = as_bf16x8(ld16(&sK[(t * 16 + fr) * LK + ks * 32 + g * 8]));
        s[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], s[t], 0, 0, 0);
      }
    }
    // Scores stay unscaled: the running max is kept in the scaled (log2)
    // domain and a probability is one FMA and one exp2. Only a block that
    // reaches past this wave's first query or the sequence end is masked.
    float bmax = -INFINITY;
    if (k0 + KB - 1 > qw0 || k0 + KB > len) {  // uniform across the wave
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = k0 + t * 16 + g * 4 + e;
          if (key > qrow || key >= len) s[t][e] = -INFINITY;
          bmax = fmaxf(bmax, s[t][e]);
        }
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) bmax = fmaxf(bmax, s[t][e]);
    }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    // finite: every wave processes block 0 and every query sees key 0
    const float m_new = fmaxf(m_run, bmax * scale_log2);
    const float corr = fast_exp2(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p = fast_exp2(__builtin_fmaf(s[t][e], scale_log2, -m_new));
        s[t][e] = p;
        psum += p;
      }
    l_run = l_run * corr + psum;
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[i] *= corr;

#pragma unroll
    for (int st = 0; st < 2; ++st) {
      pack8 pb;
      pb.w[0] = pack2bf(s[2 * st][0], s[2 * st][1]);
      pb.w[1] = pack2bf(s[2 * st][2], s[2 * st][3]);
      pb.w[2] = pack2bf(s[2 * st + 1][0], s[2 * st + 1][1]);
      pb.w[3] = pack2bf(s[2 * st + 1][2], s[2 * st + 1][3]);
      const bf16x8_v pf = as_bf16x8(pb);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        // rows of keys 32 st + 4g + (fr / 4) and 32 st + 16 + 4g + (fr / 4),
        // columns 16 dt + 4 (fr % 4) .. + 3: lane (fr, g) receives column
        // 16 dt + fr of keys 32 st + 4g + 0..3 and 32 st + 16 + 4g + 0..3
        const bf16_t* vp = &sV[(st * 32 + 4 * g + (fr >> 2)) * LV + dt * 16 + 4 * (fr & 3)];
        const s16x4_v v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4_v*)(vp));
        const s16x4_v v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) s16x4_v*)(vp + 16 * LV));
        const bf16x8_v vb = __builtin_bit_cast(
            bf16x8_v, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, pf, o[dt], 0, 0, 0);
      }
    }
  }

  if constexpr (KS == 2) {
    // odd-block waves hand (max, sum, output) to the even-block waves, lane by lane
    __shared__ float s_m[NW][64], s_l[NW][64];
    __shared__ f32x4_v s_o[NW][D / 16][64];
    __syncthreads();
    if (part == 1) {
      s_m[wave][lane] = m_run;
      s_l[wave][lane] = l_run;
#pragma unroll
      for (int i = 0; i < D / 16; ++i) s_o[wave][i][lane] = o[i];
    }
    __syncthreads();
    if (part == 1) return;
    const float m1 = s_m[wave][lane], l1 = s_l[wave][lane];
    const float m = fmaxf(m_run, m1);  // finite: the even half always has block 0
    const float c0 = fast_exp2(m_run - m), c1 = fast_exp2(m1 - m);  // m1 = -inf gives 0
    l_run = l_run * c0 + l1 * c1;
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[i] = o[i] * c0 + s_o[wave][i][lane] * c1;
  }

  float l_tot = l_run + __shfl_xor(l_run, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  if (qrow >= len) return;
  const float inv = 1.0f / l_tot;
  bf16_t* orow = a.out + (int64_t)(base + qrow) * a.ldo + h * D;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    uint2 w;
    w.x = pack2bf(o[dt][0] * inv, o[dt][1] * inv);
    w.y = pack2bf(o[dt][2] * inv, o[dt][3] * inv);
    *reinterpret_cast<uint2*>(orow + dt * 16 + g * 4) = w;
  }
}

hipError_t attn_prefill(const AttnPrefillArgs& a, hipStream_t s, LaunchInfo* info) {
  if (a.n_tiles <= 0) return hipSuccess;
  if ((a.D != 64 && a.D != 128) || a.n_kv_heads <= 0 || a.n_heads % a.n_kv_heads) return hipErrorInvalidValue;
  if ((a.ld % 8) || (a.ldo % 4) || a.q_tile != 16 * a.waves || (a.waves != 4 && a.waves != 8))
    return hipErrorInvalidValue;
  const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)a.D));
  dim3 grid(a.n_tiles, a.n_heads);
  // 4-wave tiles that fit one workgroup per CU take the key split (8 waves)
  static int cus = 0;
  if (!cus) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      cus = 1;
  }
  const bool ks = a.waves == 4 && (int64_t)a.n_tiles * a.n_heads <= cus;
  if (a.D == 128 && a.waves == 8)
    hipLaunchKernelGGL((attn_prefill_kernel<128, 8, 1>), grid, dim3(512), 0, s, a, scale_log2);
  else if (a.D == 128 && ks)
    hipLaunchKernelGGL((attn_prefill_kernel<128, 4, 2>), grid, dim3(512), 0, s, a, scale_log2);
  else if (a.D == 128)
    hipLaunchKernelGGL((attn_prefill_kernel<128, 4, 1>), grid, dim3(256), 0, s, a, scale_log2);
  else if (a.waves == 8)
    hipLaunchKernelGGL((attn_prefill_kernel<64, 8, 1>), grid, dim3(512), 0, s, a, scale_log2);
  else if (ks)
    hipLaunchKernelGGL((attn_prefill_kernel<64, 4, 2>), grid, dim3(512), 0, s, a, scale_log2);
  else
    hipLaunchKernelGGL((attn_prefill_kernel<64, 4, 1>), grid, dim3(256), 0, s, a, scale_log2);
  if (info) {
    info->name = a.D == 128 ? "attn_prefill_d128" : "attn_prefill_d64";
    info->flops = a.flops;
    info->bytes = 0;
  }
  return hipGetLastError();
}

int attn_prefill_waves(int64_t tiles_of_128, int n_heads) {
  return tiles_of_128 * n_heads >= 512 ? 8 : 4;
}

// ------------------------------------------------------------------- decode
//
// The context of a sequence is cut into fixed 128-token splits; one
// workgroup per (split, kv head, sequence). D/8 lanes share a token (one
// 16-byte chunk of its key and value rows each), so 256 threads cover
// 2048/D tokens per pass and every thread sees 8 (D = 128) or 4 (D = 64)
// tokens of the split. Per
// group of 4 tokens a thread forms the G scores (partial dot products summed
// over the token's lanes with DPP row operations), then updates its online
// softmax once: new max, one rescale of the accumulators, four
// probabilities. The token slots of a wave are merged with cross-row lane
// swaps, the four waves through LDS, in a fixed order.
//
// Each split leaves, per query head, the unnormalised P V, the max score
// (log2 domain) and the sum of exp2(score - max); a second kernel merges
// the splits in split order with a running max, so the result does not
// depend on which split ends when.

// Sum over the 16 lanes of a DPP row (all lanes get the sum). Each step adds
// a lane permutation that pairs lanes holding disjoint partial sums.
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));   // quad_perm 1,0,3,2
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));   // quad_perm 2,3,0,1
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, true));  // row_half_mirror
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, true));  // row_mirror
  return v;
}
// Sum over 8 lanes (lanes 8k..8k+7 of a row).
__device__ __forceinline__ float row8_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, true));
  return v;
}

// Lanes i and i ^ 8 of each row (row_ror:8), rows 2k and 2k + 1
// (permlane16 swap) and the two halves of the wave (permlane32 swap): the
// operands reach every lane of a group in the same order, so all of them get
// the same bits.
__device__ __forceinline__ float xor8_val(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xF, 0xF, true));
}
template <typename Op>
__device__ __forceinline__ float rows_pair(float v, Op op) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return op(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
template <typename Op>
__device__ __forceinline__ float halves_pair(float v, Op op) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return op(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// op over the token slots of a wave (lanes c + LPT j, j = 0 .. 64 / LPT - 1)
template <int LPT, typename Op>
__device__ __forceinline__ float over_slots(float v, Op op) {
  if constexpr (LPT == 8) v = op(v, xor8_val(v));
  return halves_pair(rows_pair(v, op), op);
}

constexpr int kRawBuffer = 0x00020000;   // raw buffer, 32-bit data format
__device__ __forceinline__ float ld_part(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
}

// Merge the n_splits partials of one query head (row r of ro / rml holds
// split r) in split order with a running max; 8 splits are loaded together.
// Splits [0, n_valid) of a row are merged in split order. The loads cover
// [0, n_load) (n_load >= n_valid, rows that exist in the buffer) and do not
// depend on n_valid, so they go out without waiting for the context length;
// rows past n_valid may hold anything and are dropped by selects.
template <int D>
__device__ __forceinline__ float merge_splits(__amdgpu_buffer_rsrc_t ro, __amdgpu_buffer_rsrc_t rml,
                                              int row0, int n_load, int n_valid, int d) {
  float M = -INFINITY, L = 0.f, O = 0.f;
  for (int s0 = 0; s0 < n_load; s0 += 8) {
    float ms[8], ls[8], os[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {  // past n_load: re-read the last row, then ignore
      const int row = row0 + min(s0 + u, n_load - 1);
      ms[u] = ld_part(rml, row * 8);
      ls[u] = ld_part(rml, row * 8 + 4);
      os[u] = ld_part(ro, (row * D + d) * 4);
    }
    // branch-free, so that all 24 loads are in flight together
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const bool ok = s0 + u < n_valid && ms[u] != -INFINITY;
      const float mn = ok ? fmaxf(M, ms[u]) : M;
      const float wo = ok ? fast_exp2(M - mn) : 1.f, wn = ok ? fast_exp2(ms[u] - mn) : 0.f;
      O = ok ? O * wo + os[u] * wn : O;
      L = ok ? L * wo + ls[u] * wn : L;
      M = mn;
    }
  }
  return O / L;
}

// Rotate-half RoPE of one 16-byte chunk (8 consecutive elements of a head)
// whose partner chunk (the elements D/2 away) sits in lane ^ (LPT / 2): the
// first half's lanes get x1 c - x2 s, the second half's x2 c + x1 s, in
// float32, rounded to bf16 (the arithmetic and rounding of rope_kv). Every
// lane of the wave must call it.
template <int LPT>
__device__ __forceinline__ pack8 rope_chunk(const pack8& x, bool first, const float (&cs)[8],
                                            const float (&sn)[8]) {
  pack8 y;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t pw = __shfl_xor(x.w[e], LPT / 2, 64);
    const float o0 = lo_bf(x.w[e]), o1 = hi_bf(x.w[e]), p0 = lo_bf(pw), p1 = hi_bf(pw);
    float y0, y1;
    if (first) {
      y0 = rope_first(o0, p0, cs[2 * e], sn[2 * e]);
      y1 = rope_first(o1, p1, cs[2 * e + 1], sn[2 * e + 1]);
    } else {
      y0 = rope_second(p0, o0, cs[2 * e], sn[2 * e]);
      y1 = rope_second(p1, o1, cs[2 * e + 1], sn[2 * e + 1]);
    }
    y.w[e] = pack2bf(y0, y1);
  }
  return y;
}

template <int D, int G, bool ROPE>
__global__ __launch_bounds__(256) void attn_decode_split_kernel(AttnDecodeArgs a, float scale_log2) {

  constexpr int LPT = D / 8;        // lanes per token
  constexpr int TPP = 256 / LPT;    // tokens per pass
  constexpr int PASSES = kDecodeSplit / TPP;
  constexpr int UNR = PASSES < 4 ? PASSES : 4;
  static_assert(PASSES % UNR == 0, "split/pass mismatch");
  static_assert(LPT == 16 || LPT == 8, "head dim 128 or 64");
  static_assert(TPP == 16 || TPP == 32, "one or two cache blocks per pass");
  constexpr int BPS = kDecodeSplit / 16;  // cache blocks per split
  static_assert(BPS * 16 == kDecodeSplit && PASSES * TPP == kDecodeSplit, "split of whole blocks");
  __shared__ float s_ml[4][G][2];
  __shared__ float s_acc[4][G][D];

  const int split = blockIdx.x, kh = blockIdx.y, b = blockIdx.z;
  // the split's block-table entries are loaded together with the context
  // length: one round trip before the key/value loads instead of two
  const int32_t* bt = a.block_table + (int64_t)b * a.max_blocks;
  int phys[BPS];
#pragma unroll
  for (int j = 0; j < BPS; ++j) phys[j] = bt[min(split * BPS + j, a.max_blocks - 1)];  // past: unused
  const int ctx = a.ctx[b];
#pragma unroll
  for (int j = 0; j < BPS; ++j) asm volatile("" ::"s"(phys[j]));  // not sunk below the branch
  const int t_begin = split * kDecodeSplit;
  if (t_begin >= ctx) return;  // uniform across the workgroup
  const int tid = threadIdx.x, tl = tid / LPT, c = tid % LPT;
  const int h0 = kh * G;
  const int64_t kv_stride = (int64_t)a.n_kv_heads * 16 * D;  // K block -> V block

  // the new token (fused RoPE) sits at offset t_new of this split when that
  // is below the split length
  const int t_new = ctx - 1 - t_begin;  // >= 0; uniform
  const bool has_new = ROPE && t_new < kDecodeSplit;
  const bf16_t* qrow = a.q + (int64_t)b * a.ldq;

  // all key and value loads of the split go out first (non-temporal: each
  // cached byte is read once per step)
  pack8 kv[PASSES], vv[PASSES];
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int tok = t_begin + p * TPP + tl;
    kv[p] = zero8();
    vv[p] = zero8();
    if (tok < ctx) {
      const int ph = TPP == 16 ? phys[p] : ((tl >> 4) ? phys[2 * p + 1] : phys[2 * p]);
      const bf16_t* kp = a.pool + ((int64_t)ph * 2 * a.n_kv_heads + kh) * 16 * D +
                         (tok & 15) * D + c * 8;
      int64_t vo = kv_stride;
      if (ROPE && tok == ctx - 1) {  // not in the pool yet: the projection's rows
        kp = qrow + (int64_t)(a.n_heads + kh) * D + c * 8;
        vo = (int64_t)a.n_kv_heads * D;
      }
      kv[p] = ld16_nt(kp);
      vv[p] = ld16_nt(kp + vo);
    }
  }
  float cs[8], sn[8];
  const bool first = c < LPT / 2;
  if constexpr (ROPE) {
    const int j = (c % (LPT / 2)) * 8;
    const float* ct = a.cos_t + (int64_t)(ctx - 1) * (D / 2) + j;
    const float* st = a.sin_t + (int64_t)(ctx - 1) * (D / 2) + j;
#pragma unroll
    for (int e = 0; e < 8; e += 4) {
      const float4 cv = *reinterpret_cast<const float4*>(ct + e);
      const float4 sv = *reinterpret_cast<const float4*>(st + e);
      cs[e] = cv.x;
      cs[e + 1] = cv.y;
      cs[e + 2] = cv.z;
      cs[e + 3] = cv.w;
      sn[e] = sv.x;
      sn[e + 1] = sv.y;
      sn[e + 2] = sv.z;
      sn[e + 3] = sv.w;
    }
  }
  float q[G][8];
#pragma unroll
  for (int gg = 0; gg < G; ++gg) {
    pack8 v = ld16(qrow + (h0 + gg) * D + c * 8);
    if constexpr (ROPE) v = rope_chunk<LPT>(v, first, cs, sn);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      q[gg][2 * e] = lo_bf(v.w[e]);
      q[gg][2 * e + 1] = hi_bf(v.w[e]);
    }
  }
  if (has_new) {
    // rotate the new key (the whole wave takes part), use it for the scores
    // and append key and value to the cache
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      if (p != t_new / TPP) continue;
      const pack8 kr = rope_chunk<LPT>(kv[p], first, cs, sn);
      if (tl == t_new % TPP) {
        kv[p] = kr;
        const int blk = t_new / 16;
        int ph = phys[0];
#pragma unroll
        for (int j = 1; j < BPS; ++j) ph = blk == j ? phys[j] : ph;
        bf16_t* kd = a.pool_w + ((int64_t)ph * 2 * a.n_kv_heads + kh) * 16 * D +
                     ((ctx - 1) & 15) * D + c * 8;
        st16(kd, kr);
        st16(kd + kv_stride, vv[p]);
      }
    }
  }
  const int wave = tid >> 6;
  const auto fmax_op = [](float x, float y) { return fmaxf(x, y); };
  const auto add_op = [](float x, float y) { return x + y; };
  // partials of this (sequence, kv head): [G][max_splits][D] and [G][max_splits][2]
  const int64_t base = ((int64_t)b * a.n_heads + h0) * a.max_splits;

  {
    float m[G], l[G], acc[G][8];
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      m[gg] = -INFINITY;
      l[gg] = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[gg][e] = 0.f;
    }
#pragma unroll
    for (int p0 = 0; p0 < PASSES; p0 += UNR) {
      float sc[UNR][G];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const bool ok = t_begin + (p0 + u) * TPP + tl < ctx;
        float kf[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kf[2 * e] = lo_bf(kv[p0 + u].w[e]);
          kf[2 * e + 1] = hi_bf(kv[p0 + u].w[e]);
        }
#pragma unroll
        for (int gg = 0; gg < G; ++gg) {
          float d = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) d += q[gg][e] * kf[e];
          d = LPT == 16 ? row16_sum(d) : row8_sum(d);
          sc[u][gg] = ok ? d * scale_log2 : -INFINITY;
        }
      }
#pragma unroll
      for (int gg = 0; gg < G; ++gg) {
        float mx = m[gg];
#pragma unroll
        for (int u = 0; u < UNR; ++u) mx = fmaxf(mx, sc[u][gg]);
        if (mx == -INFINITY) continue;  // no valid token yet for this slot
        const float corr = fast_exp2(m[gg] - mx);
        l[gg] *= corr;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[gg][e] *= corr;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          const float pr = sc[u][gg] == -INFINITY ? 0.f : fast_exp2(sc[u][gg] - mx);
          l[gg] += pr;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[gg][2 * e] += pr * lo_bf(vv[p0 + u].w[e]);
            acc[gg][2 * e + 1] += pr * hi_bf(vv[p0 + u].w[e]);
          }
        }
        m[gg] = mx;
      }
    }

    // token slots of the wave -> one (lanes 0 .. LPT - 1 keep it)
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      const float M = over_slots<LPT>(m[gg], fmax_op);
      const float w = m[gg] == -INFINITY ? 0.f : fast_exp2(m[gg] - M);
      const float L = over_slots<LPT>(l[gg] * w, add_op);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[gg][e] = over_slots<LPT>(acc[gg][e] * w, add_op);
      if (tid % 64 < LPT) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s_acc[wave][gg][c * 8 + e] = acc[gg][e];
        if (c == 0) {
          s_ml[wave][gg][0] = M;
          s_ml[wave][gg][1] = L;
        }
      }
    }
    __syncthreads();
    for (int i = tid; i < G * D; i += 256) {
      const int gg = i / D, d = i % D;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) M = fmaxf(M, s_ml[w][gg][0]);
      float L = 0.f, O = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float mw = s_ml[w][gg][0];
        if (mw == -INFINITY) continue;
        const float f = fast_exp2(mw - M);
        L += s_ml[w][gg][1] * f;
        O += s_acc[w][gg][d] * f;
      }
      const int64_t row = base + gg * a.max_splits + split;
      a.part_o[row * D + d] = O;
      if (d == 0) {
        a.part_ml[row * 2] = M;
        a.part_ml[row * 2 + 1] = L;
      }
    }
  }
}

// MFMA form of the split kernel for grouped-query heads (G >= 2, D = 128).
// Wave w takes tokens 32w .. 32w + 31 of the split (two cache blocks). The
// keys and values are read with whole-row loads (each instruction covers 4
// rows of 256 bytes, lane l taking chunk l % 16 of row l / 16; the MFMA
// operand order, 64 bytes of each of 16 rows per instruction, streamed
// 15-17% slower on MI355X) and staged row-major through the wave's LDS
// buffer: first the keys, read back in operand order, then the values.
// Scores are formed transposed, S^T = K Q^T, with 16x16x32 MFMAs: the keys
// on the rows (lane (r, g) holds key r of a block, d-chunk g of each 32-d
// step) and the G query heads of the kv head on the columns (the other
// columns zero), so lane (r, g) ends with the scores of keys 4g .. 4g+3 (and
// 16 + 4g .. 16 + 4g + 3) for query head r. P V^T reads its V^T fragments
// with transposing LDS reads (as the prefill kernel does); the
// probabilities are the B operand exactly as the score MFMAs left them.
// With fused RoPE the rotation pairs (d, d + D/2) sit in one lane. The
// waves' partial results are merged through LDS in wave order; each wave's
// partial reuses its own (by then consumed) value buffer.
typedef short s16x4_dv __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void rope_pair(pack8& x1, pack8& x2, const float* cs, const float* sn) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float a0 = lo_bf(x1.w[e]), a1 = hi_bf(x1.w[e]);
    const float b0 = lo_bf(x2.w[e]), b1 = hi_bf(x2.w[e]);
    const float c0 = cs[2 * e], c1 = cs[2 * e + 1], s0 = sn[2 * e], s1 = sn[2 * e + 1];
    x1.w[e] = pack2bf(rope_first(a0, b0, c0, s0), rope_first(a1, b1, c1, s1));
    x2.w[e] = pack2bf(rope_second(a0, b0, c0, s0), rope_second(a1, b1, c1, s1));
  }
}

template <int G, bool ROPE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void attn_decode_gqa_kernel(
    AttnDecodeArgs a, float scale_log2) {
  constexpr int D = 128;
  static_assert(G >= 2 && G <= 16, "the query heads of a kv head fit the 16 MFMA columns");
  static_assert(kDecodeSplit == 128, "four waves of two cache blocks");
  constexpr int KS = D / 32;      // 32-d steps of the score MFMAs; value chunks per lane per block
  constexpr int DT = D / 16;      // 16-row tiles of d in the P V MFMAs
  constexpr int LV = D + 16;      // padded V row (transposing reads on distinct banks)
  constexpr int BPS = kDecodeSplit / 16;
  __shared__ __attribute__((aligned(16))) bf16_t sV[4][32 * LV];
  __shared__ float s_ml[4][G][2];
  // wave w's partial output [G][D] reuses its own value buffer (read by
  // that wave only, and consumed before the partial is written)
  static_assert(G * D * 4 <= 32 * LV * 2, "a wave's partial fits its value buffer");
  const auto s_acc = [&](int w) { return reinterpret_cast<float*>(sV[w]); };

  const int split = blockIdx.x, kh = blockIdx.y, b = blockIdx.z;
  const int32_t* bt = a.block_table + (int64_t)b * a.max_blocks;
  int phys[BPS];
#pragma unroll
  for (int j = 0; j < BPS; ++j) phys[j] = bt[min(split * BPS + j, a.max_blocks - 1)];  // past: unused
  const int ctx = a.ctx[b];
#pragma unroll
  for (int j = 0; j < BPS; ++j) asm volatile("" ::"s"(phys[j]));  // not sunk below the branch
  const int t_begin = split * kDecodeSplit;
  if (t_begin >= ctx) return;  // uniform across the workgroup
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int fr = lane & 15, g = lane >> 4;
  const int h0 = kh * G;
  const int64_t kv_stride = (int64_t)a.n_kv_heads * 16 * D;  // K block -> V block
  const bf16_t* qrow = a.q + (int64_t)b * a.ldq;
  const int tb = t_begin + wave * 32;  // first token of this wave

  pack8 kf[2][KS], ck[2][4], cv[2][4], qf[KS];
  bool is_new[2];
  int ph[2];
  // whole-row loads: instruction i of block t takes rows 4i .. 4i + 3 of the
  // block (lane l: row 4i + l / 16, 16-byte chunk l % 16); all of them go
  // out first (non-temporal: each cached byte is read once per step)
  const int crow = lane >> 4, cch = lane & 15;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int blk = wave * 2 + t;
    int p = phys[0];
#pragma unroll
    for (int j = 1; j < BPS; ++j) p = blk == j ? phys[j] : p;
    ph[t] = p;
    is_new[t] = ROPE && tb + 16 * t + fr == ctx - 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + crow, tok = tb + 16 * t + r;
      const bf16_t* krow = a.pool + ((int64_t)p * 2 * a.n_kv_heads + kh) * 16 * D + r * D;
      const bf16_t* vrow = krow + kv_stride;
      if (ROPE && tok == ctx - 1) {  // not in the pool yet: the projection's rows
        krow = qrow + (int64_t)(a.n_heads + kh) * D;
        vrow = qrow + (int64_t)(a.n_heads + a.n_kv_heads + kh) * D;
      }
      ck[t][i] = tok < ctx ? ld16_nt(krow + cch * 8) : zero8();
      cv[t][i] = tok < ctx ? ld16_nt(vrow + cch * 8) : zero8();
    }
  }
  // keys row-major into this wave's buffer (key 16 t + row), read back in
  // the score MFMAs' operand order; then the values over them (one wave's
  // LDS operations run in order)
  bf16_t* sv = sV[wave];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<pack8*>(sv + (16 * t + 4 * i + crow) * LV + cch * 8) = ck[t][i];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kf[t][ks] = *reinterpret_cast<const pack8*>(sv + (16 * t + fr) * LV + ks * 32 + g * 8);
  asm volatile("" ::: "memory");  // the key reads before the value stores
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<pack8*>(sv + (16 * t + 4 * i + crow) * LV + cch * 8) = cv[t][i];
  if constexpr (ROPE) {  // the new token's value into its pool slot (its key below, rotated)
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * i + crow;
        if (tb + 16 * t + r == ctx - 1)
          st16(a.pool_w + ((int64_t)ph[t] * 2 * a.n_kv_heads + kh) * 16 * D + kv_stride + r * D + cch * 8,
               cv[t][i]);
      }
  }
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qf[ks] = fr < G ? ld16(qrow + (h0 + fr) * D + ks * 32 + g * 8) : zero8();
  if constexpr (ROPE) {
    // lane (r, g) holds d = 32 ks + 8 g + e; its pair partners d + D/2 are
    // chunk ks + KS/2 of the same lane
    const float* ct = a.cos_t + (int64_t)(ctx - 1) * (D / 2);
    const float* st = a.sin_t + (int64_t)(ctx - 1) * (D / 2);
#pragma unroll
    for (int ks = 0; ks < KS / 2; ++ks) {
      float cs[8], sn[8];
#pragma unroll
      for (int e = 0; e < 8; e += 4) {
        const float4 c4 = *reinterpret_cast<const float4*>(ct + ks * 32 + g * 8 + e);
        const float4 s4 = *reinterpret_cast<const float4*>(st + ks * 32 + g * 8 + e);
        cs[e] = c4.x;
        cs[e + 1] = c4.y;
        cs[e + 2] = c4.z;
        cs[e + 3] = c4.w;
        sn[e] = s4.x;
        sn[e + 1] = s4.y;
        sn[e + 2] = s4.z;
        sn[e + 3] = s4.w;
      }
      rope_pair(qf[ks], qf[ks + KS / 2], cs, sn);
#pragma unroll
      for (int t = 0; t < 2; ++t)
        if (is_new[t]) rope_pair(kf[t][ks], kf[t][ks + KS / 2], cs, sn);
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
      if (is_new[t]) {  // append the rotated key to the cache
        bf16_t* kd = a.pool_w + ((int64_t)ph[t] * 2 * a.n_kv_heads + kh) * 16 * D + fr * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) st16(kd + ks * 32 + g * 8, kf[t][ks]);
      }
  }

  // S^T: lane (r, g) gets keys tb + 16 t + 4g + j of query head r
  f32x4_v s[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    s[t] = f32x4_v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      s[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[t][ks]), as_bf16x8(qf[ks]), s[t], 0, 0, 0);
  }
  float m = -INFINITY;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (tb + 16 * t + 4 * g + j >= ctx) s[t][j] = -INFINITY;
      m = fmaxf(m, s[t][j]);
    }
  m = fmaxf(m, __shfl_xor(m, 16, 64));
  m = fmaxf(m, __shfl_xor(m, 32, 64));
  const float ms = m * scale_log2;  // running max in the scaled (log2) domain
  float l = 0.f;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      s[t][j] = m == -INFINITY ? 0.f : fast_exp2(__builtin_fmaf(s[t][j], scale_log2, -ms));
      l += s[t][j];
    }
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  pack8 pk;
  pk.w[0] = pack2bf(s[0][0], s[0][1]);
  pk.w[1] = pack2bf(s[0][2], s[0][3]);
  pk.w[2] = pack2bf(s[1][0], s[1][1]);
  pk.w[3] = pack2bf(s[1][2], s[1][3]);
  const bf16x8_v pf = as_bf16x8(pk);
  asm volatile("" ::: "memory");  // the value stores (this wave's) before the fragment reads
  // O^T = V^T P^T: lane (r, g) gets rows d = 16 dt + 4g + j of query head r
  f32x4_v o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    const bf16_t* vp = sv + (4 * g + (fr >> 2)) * LV + dt * 16 + 4 * (fr & 3);
    const s16x4_dv v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_dv*)(vp));
    const s16x4_dv v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_dv*)(vp + 16 * LV));
    const bf16x8_v vb =
        __builtin_bit_cast(bf16x8_v, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
    o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, pf, f32x4_v{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
  }

  if (fr < G) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      *reinterpret_cast<f32x4_v*>(s_acc(wave) + fr * D + dt * 16 + 4 * g) = o[dt];
    if (g == 0) {
      s_ml[wave][fr][0] = ms;
      s_ml[wave][fr][1] = l;
    }
  }
  __syncthreads();
  // partials of this (sequence, kv head): [G][max_splits][D] and [G][max_splits][2]
  const int64_t base = ((int64_t)b * a.n_heads + h0) * a.max_splits;
  for (int i = tid; i < G * D; i += 256) {
    const int gg = i / D, d = i % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_ml[w][gg][0]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float mw = s_ml[w][gg][0];
      if (mw == -INFINITY) continue;
      const float f = fast_exp2(mw - M);
      L += s_ml[w][gg][1] * f;
      O += s_acc(w)[gg * D + d] * f;
    }
    const int64_t row = base + gg * a.max_splits + split;
    a.part_o[row * D + d] = O;
    if (d == 0) {
      a.part_ml[row * 2] = M;
      a.part_ml[row * 2 + 1] = L;
    }
  }
}

// Merge of the splits of every (query head, sequence).
template <int D>
__global__ __launch_bounds__(D) void attn_decode_combine_kernel(AttnDecodeArgs a) {
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int n_splits = (a.ctx[b] + kDecodeSplit - 1) / kDecodeSplit;
  const int64_t base = ((int64_t)b * a.n_heads + h) * a.max_splits;
  const __amdgpu_buffer_rsrc_t ro =
      __builtin_amdgcn_make_buffer_rsrc(a.part_o + base * D, 0, a.max_splits * D * 4, kRawBuffer);
  const __amdgpu_buffer_rsrc_t rml =
      __builtin_amdgcn_make_buffer_rsrc(a.part_ml + base * 2, 0, a.max_splits * 8, kRawBuffer);
  a.out[(int64_t)b * a.ldo + h * D + d] =
      f2bf(merge_splits<D>(ro, rml, 0, a.call_splits, n_splits, d));
}

namespace {
template <int D, int G>
void launch_split(const AttnDecodeArgs& a, float sl, hipStream_t s) {
  dim3 grid(a.call_splits, a.n_kv_heads, a.B);
  static const char* force = getenv("HS_DECODE_ATTN");  // "valu" (tuning only)
  if constexpr (D == 128 && G >= 2) {
    if (!(force && strcmp(force, "valu") == 0)) {
      if (a.pool_w)
        hipLaunchKernelGGL((attn_decode_gqa_kernel<G, true>), grid, dim3(256), 0, s, a, sl);
      else
        hipLaunchKernelGGL((attn_decode_gqa_kernel<G, false>), grid, dim3(256), 0, s, a, sl);
      return;
    }
  }
  if (a.pool_w)
    hipLaunchKernelGGL((attn_decode_split_kernel<D, G, true>), grid, dim3(256), 0, s, a, sl);
  else
    hipLaunchKernelGGL((attn_decode_split_kernel<D, G, false>), grid, dim3(256), 0, s, a, sl);
}
template <int D>
hipError_t launch_split_g(const AttnDecodeArgs& a, int G, float sl, hipStream_t s) {
  switch (G) {
    case 1: launch_split<D, 1>(a, sl, s); break;
    case 2: launch_split<D, 2>(a, sl, s); break;
    case 4: launch_split<D, 4>(a, sl, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t attn_decode(const AttnDecodeArgs& a, hipStream_t s, LaunchInfo* info) {
  if (a.B <= 0) return hipSuccess;
  if ((a.D != 64 && a.D != 128) || a.n_kv_heads <= 0 || a.n_heads % a.n_kv_heads) return hipErrorInvalidValue;
  if (a.call_splits <= 0 || a.call_splits > a.max_splits || (a.ldq % 8)) return hipErrorInvalidValue;
  if (a.pool_w && (!a.cos_t || !a.sin_t || a.max_pos <= 0 || a.pool_w != a.pool))
    return hipErrorInvalidValue;
  // byte offsets of one (query head, sequence)'s partials fit 32 bits
  if ((int64_t)a.max_splits * a.D * 4 >= (1ll << 31)) return hipErrorInvalidValue;
  const int G = a.n_heads / a.n_kv_heads;
  const float sl = (float)(1.4426950408889634 / sqrt((double)a.D));
  hipError_t e = a.D == 128 ? launch_split_g<128>(a, G, sl, s) : launch_split_g<64>(a, G, sl, s);
  if (e != hipSuccess) return e;
  dim3 grid(a.n_heads, a.B);
  if (a.D == 128)
    hipLaunchKernelGGL(attn_decode_combine_kernel<128>, grid, dim3(128), 0, s, a);
  else
    hipLaunchKernelGGL(attn_decode_combine_kernel<64>, grid, dim3(64), 0, s, a);
  if (info) {
    info->name = "attn_decode";
    info->flops = 0;
    info->bytes = a.kv_bytes;
  }
  return hipGetLastError();
}

}  // namespace hs
