// Host-side launchers of the engine's HIP kernels. Every launcher checks the
// shapes its kernel assumes and returns hipErrorInvalidValue instead of
// launching when they do not hold.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hs {

typedef uint16_t bf16_t;

// Epilogues of Y[m][n] = sum_k X[m][k] * W[n][k] (fp32 accumulation).
enum Epi : int {
  EPI_STORE = 0,   // Y = bf16(acc)
  EPI_RESID = 1,   // Y = bf16(R + acc); R may alias Y
  EPI_SWIGLU = 2,  // W rows interleave 16 gate / 16 up rows; Y[m][f] = bf16(silu(g) * u), width N/2
  EPI_F32 = 3,     // Y = acc as float32
  EPI_QKV_ROPE = 4  // QKV projection: Y as EPI_STORE with q and k rotated (RoPE), k and v
                    // also appended to the paged KV pool (fields rope_* below)
};

struct GemmArgs {
  const bf16_t* X; int64_t ldx;  // [M][K] activations, row stride ldx elements
  const bf16_t* W;               // [N][K] weights in the tiled matrix format
  void* Y; int64_t ldy;          // output, row stride ldy elements (of its type)
  const bf16_t* R; int64_t ldr;  // residual input for EPI_RESID
  int M, N, K;
  // Optional workspace for split-k tiles (stream-K launches): fp32 partial
  // tiles and per-tile arrival counters, which must be zero before the first
  // launch and are left at zero by every launch. Launches that share a
  // workspace must not overlap in time.
  float* part = nullptr; int64_t part_floats = 0;
  uint32_t* flags = nullptr; int64_t flags_n = 0;
  // Optional RMSNorm of the rows of X with this gain (M <= 16, K % 64 == 0):
  // the product is then of rmsnorm(X) * gain, X being the raw rows.
  const bf16_t* norm_gain = nullptr; float norm_eps = 0.f;
  // QKV projection with head-interleaved q and k rows: when rope_q_cols +
  // rope_kv_cols > 0, the first rope_q_cols (q heads) and next rope_kv_cols (k
  // heads) rows of W are stored per head as 32-row groups, 16 rows of the
  // head's first half followed by the matching 16 rows of its second half
  // (RoPE partners), so that a 32-row output pair holds both partners. Every
  // store puts the columns back in head order. EPI_QKV_ROPE additionally
  // rotates q and k (rotate-half RoPE at pos[m], tables [max_pos][D/2]) and
  // writes k and v to token m's slot of the pool [blocks][2][n_kv][16][D]
  // (slot < 0: no append); the v rows (the last rope_kv_cols) keep their order.
  int rope_q_cols = 0, rope_kv_cols = 0, rope_d = 0;
  const int32_t* rope_pos = nullptr; const int32_t* rope_slot = nullptr;
  const float* rope_cos = nullptr; const float* rope_sin = nullptr;
  int rope_max_pos = 0;
  bf16_t* rope_pool = nullptr;
};

// Describes what was launched (for timing).
struct LaunchInfo {
  const char* name;
  double flops;
  double bytes;
};

hipError_t gemm(const GemmArgs& a, int epi, hipStream_t s, LaunchInfo* info);

hipError_t embed(const int32_t* tok, const bf16_t* E, int vocab, int hidden, int n_tok,
                 bf16_t* out, hipStream_t s, LaunchInfo* info);

// out[r] = rmsnorm(x[rows ? rows[r] : r]) * g
hipError_t rmsnorm(const bf16_t* x, int64_t ldx, const int32_t* rows, int n_rows, int hidden,
                   const bf16_t* g, float eps, bf16_t* out, int64_t ldo, hipStream_t s,
                   LaunchInfo* info);

struct RopeKvArgs {
  bf16_t* qkv; int64_t ld;       // [T][ld]: q heads, k heads, v heads
  const int32_t* pos;            // [T] position of each token
  const int32_t* slot;           // [T] physical KV slot (block * 16 + offset)
  const float* cos_t; const float* sin_t;  // [max_pos][D/2]
  bf16_t* pool;                  // this layer's pool [blocks][2][n_kv][16][D]
  int T, n_heads, n_kv_heads, D, max_pos;
};
hipError_t rope_kv(const RopeKvArgs& a, hipStream_t s, LaunchInfo* info);

struct AttnPrefillArgs {
  const bf16_t* qkv; int64_t ld;  // post-RoPE q, k and v
  bf16_t* out; int64_t ldo;       // [T][n_heads * D]
  const int32_t* cu;              // [n_seqs + 1] token offsets
  const int32_t* tiles;           // [n_tiles][2] (sequence, first query row, multiple of q_tile)
  int n_tiles, n_heads, n_kv_heads, D;
  int waves, q_tile;              // 4 or 8 waves; q_tile = 16 * waves queries per workgroup
  double flops;                   // unmasked-pair flops, for reporting
};
hipError_t attn_prefill(const AttnPrefillArgs& a, hipStream_t s, LaunchInfo* info);
// Waves per prefill-attention workgroup for a problem with `tiles_of_128`
// 128-query tiles (summed over sequences) and n_heads heads.
int attn_prefill_waves(int64_t tiles_of_128, int n_heads);

constexpr int kDecodeSplit = 128;  // tokens per split of the decode attention

struct AttnDecodeArgs {
  const bf16_t* q; int64_t ldq;   // [B][ldq], query heads at column h * D
  const bf16_t* pool;             // layer pool [blocks][2][n_kv][16][D]
  const int32_t* block_table;     // [B][max_blocks]
  const int32_t* ctx;             // [B] cached positions including the new one
  float* part_o;                  // [B][n_heads][max_splits][D]
  float* part_ml;                 // [B][n_heads][max_splits][2]
  bf16_t* out; int64_t ldo;       // [B][n_heads * D]
  int B, n_heads, n_kv_heads, D, max_blocks, max_splits, call_splits;
  double kv_bytes;                // bytes of K/V read, for reporting
  // Fused RoPE and cache append (decode steps): when pool_w is set, q points
  // at the rows of the QKV projection before RoPE ([B][ldq]: query heads,
  // then key heads, then value heads), position ctx - 1 of each sequence is
  // the new token, whose key and value are read from those rows instead of
  // the pool; the kernel rotates the queries and the new key (the rotation
  // and bf16 rounding of rope_kv) and writes the new key and value into the
  // token's slot of pool_w (the same pool as `pool`).
  bf16_t* pool_w = nullptr;
  const float* cos_t = nullptr; const float* sin_t = nullptr;  // [max_pos][D/2]
  int max_pos = 0;
};
hipError_t attn_decode(const AttnDecodeArgs& a, hipStream_t s, LaunchInfo* info);

// Greedy token per row: lowest index of the row's maximum. part: scratch of
// n_rows * argmax_chunks(n_cols) * 2 int32.
int argmax_chunks(int n_cols);
hipError_t argmax_rows(const float* logits, int n_rows, int n_cols, int32_t* part, int32_t* out,
                       hipStream_t s, LaunchInfo* info);

// Copy `n` int32 values (n % 4 == 0, both pointers 16-byte aligned) from
// pinned host memory to device memory with system-coherent loads, and in the
// same launch `n2` more from host2 to dev2 (same rules; n2 = 0: none): the
// per-call metadata and copy descriptors of a stage, pulled by a kernel.
hipError_t meta_pull(const int32_t* host, int32_t* dev, int64_t n, hipStream_t s,
                     const int32_t* host2 = nullptr, int32_t* dev2 = nullptr, int64_t n2 = 0);

// Copy `n_units` KV units (a K block followed by its V block, unit_bytes each);
// slots at or past valid[u] are written as zero when zero_tail is set.
hipError_t kv_copy(const uint64_t* src, const uint64_t* dst, const int32_t* valid, int n_units,
                   int64_t unit_bytes, int D, int zero_tail, hipStream_t s, LaunchInfo* info);

}  // namespace hs
