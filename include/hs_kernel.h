/*
 * hs_kernel.h - single-kernel entry points of the stage engine.
 *
 * These run one of the engine's HIP kernels on caller-owned device buffers,
 * exactly as the stage forward pass launches it. They exist so that each
 * kernel can be checked against a reference and timed on its own; serving
 * goes through hs.h. All pointers are device pointers owned by the caller;
 * `stream` is a hipStream_t (NULL = the null stream). Work is asynchronous.
 * Shapes the kernel does not support return HS_EINVAL before any launch.
 */
#ifndef HS_KERNEL_H
#define HS_KERNEL_H

#include <stdint.h>

#include "hs.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Y[m][n] = epilogue(sum_k X[m][k] W[n][k]) with fp32 accumulation. X is
 * bf16 row-major with row stride ldx (elements); W is the [N][K] matrix in
 * the tiled matrix format of hs.h (hs_pack_tiled). epi: 0 store bf16; 1 add
 * the bf16 residual R (row stride ldr; may alias Y); 2 SwiGLU on gate/up rows
 * interleaved in groups of 16, Y has N/2 columns; 3 store float32. Requires
 * K % 8 == 0, N % 16 == 0 (N % 32 for SwiGLU), 16-byte aligned X, W, Y; if
 * K % 64 != 0, ldx must be at least K rounded up to 64 and the extra columns
 * of X zero. This is the projection arithmetic of every decoder layer (QKV,
 * O, gate/up, down) and of the LM head. Shapes with few output tiles split
 * their k range over workgroups; the partial sums go through a workspace
 * that the library allocates once per device (128 MiB + 256 KiB, on the
 * first call) and keeps until the process ends, so calls on one device must not
 * run concurrently. Results are deterministic: the same inputs give the same
 * bits on every call. */
hs_status hs_k_gemm(const void* X, int64_t ldx, const void* W, void* Y, int64_t ldy,
                    const void* R, int64_t ldr, int32_t M, int32_t N, int32_t K, int32_t epi,
                    void* stream);

/* The same product with the RMSNorm of X's rows folded in (the norm of
 * section 2.1's decoder layer before attention and before the FFN):
 * Y = epilogue(rmsnorm(X) W^T) with rmsnorm(x) = x / sqrt(mean(x^2) + eps) * g,
 * g a bf16 [K] gain. X holds the raw rows; every activation is multiplied
 * by the gain and rounded to bf16 on the way into the product, and each
 * output row is scaled by its 1 / RMS in float32 afterwards. For decode
 * batches: requires 1 <= M <= 16 and K % 64 == 0 (HS_EINVAL otherwise);
 * other arguments, epilogues and the workspace as hs_k_gemm. */
hs_status hs_k_gemm_rmsnorm(const void* X, int64_t ldx, const void* g, float eps, const void* W,
                            void* Y, int64_t ldy, const void* R, int64_t ldr, int32_t M,
                            int32_t N, int32_t K, int32_t epi, void* stream);

/* Causal grouped-query attention over packed sequences (the attention of the
 * prefill pass). qkv: bf16 [T][(n_heads + 2 n_kv_heads) head_dim] holding
 * post-RoPE q, k, v per token; out: bf16 [T][n_heads head_dim]; cu_seqlens:
 * HOST int32 [n_seqs + 1] token offsets (cu[0] = 0, cu[n] = T). */
hs_status hs_k_attn_prefill(const void* qkv, void* out, const int32_t* cu_seqlens,
                            int32_t n_seqs, int32_t n_heads, int32_t n_kv_heads,
                            int32_t head_dim, void* stream);

/* Attention of one new query per sequence over its paged KV cache (the
 * attention of a decode step: the keys and values cached during prefill and
 * earlier steps are reused). q: bf16 [B][ldq], query head h at column
 * h * head_dim, already rotated; pool: one layer's KV pool, bf16
 * [blocks][K | V][n_kv_heads][16][head_dim] with post-RoPE keys;
 * block_table: device int32 [B][max_blocks] (logical block -> pool block);
 * ctx: device int32 [B], cached tokens of each sequence including the new
 * one (1 <= ctx <= max_ctx); out: bf16 [B][ldo], head h at column
 * h * head_dim. max_ctx (host) sizes the launch. The context is processed in
 * fixed 128-token splits whose partial results go through a workspace that
 * the library allocates per device on first use and grows when needed
 * (calls on one device must not overlap); the call is asynchronous on
 * `stream` and deterministic. */
hs_status hs_k_attn_decode(const void* q, int64_t ldq, const void* pool,
                           const int32_t* block_table, const int32_t* ctx, void* out,
                           int64_t ldo, int32_t B, int32_t n_heads, int32_t n_kv_heads,
                           int32_t head_dim, int32_t max_blocks, int32_t max_ctx,
                           void* stream);

/* The same attention with the decode step's RoPE and cache append folded in
 * (LLM inference: the new token's key and value join the cache and every
 * later step reuses them). qkv: bf16 [B][ldqkv], the QKV projection of each
 * sequence's new token before RoPE (query heads, then key heads, then value
 * heads, head_dim columns each); the new token sits at position ctx - 1 of
 * its sequence and is NOT read from the pool: the call rotates the queries
 * and the new key by the rotate-half RoPE at that position (float32
 * arithmetic, bf16 rounding), attends over the cached tokens plus the new
 * one, and writes the rotated key and the value into the token's slot of
 * pool (block block_table[b][(ctx - 1) / 16], offset (ctx - 1) % 16), which
 * the caller must have allocated. cos_t, sin_t: device float32
 * [max_pos][head_dim / 2], cos and sin of pos * base^(-2 i / head_dim);
 * max_ctx <= max_pos. Other arguments, workspace and errors as for
 * hs_k_attn_decode. */
hs_status hs_k_attn_decode_rope(const void* qkv, int64_t ldqkv, void* pool,
                                const int32_t* block_table, const int32_t* ctx,
                                const float* cos_t, const float* sin_t, int32_t max_pos,
                                void* out, int64_t ldo, int32_t B, int32_t n_heads,
                                int32_t n_kv_heads, int32_t head_dim, int32_t max_blocks,
                                int32_t max_ctx, void* stream);

/* Greedy sampling of the first token and of every decode step (section 2.1:
 * the next token is chosen from the logits of the last position): out[r] =
 * the lowest column index c with logits[r][c] equal to the row's maximum.
 * logits: device float32 [n_rows][n_cols], row-major, 16-byte aligned;
 * out: device int32 [n_rows]. Requires n_rows >= 1 and n_cols >= 1 with
 * n_cols % 4 == 0 (HS_EINVAL otherwise). NaN entries never win; a row of
 * NaN only gives 0x7FFFFFFF. The call allocates a small device buffer for
 * the per-chunk candidates, launches the two passes on `stream`, waits for
 * them and frees the buffer. */
hs_status hs_k_argmax(const float* logits, int32_t n_rows, int32_t n_cols, int32_t* out,
                      void* stream);

/* RMSNorm of `rows` rows of width `hidden`: out = x / sqrt(mean(x^2) + eps) * g,
 * bf16 in and out, float32 arithmetic. */
hs_status hs_k_rmsnorm(const void* x, const void* g, void* out, int32_t rows, int32_t hidden,
                       float eps, void* stream);

/* hs_k_attn_decode without any device allocation, for callers that cannot
 * allocate: code under HIP graph capture, serving loops that must not call
 * hipMalloc, harnesses that forbid it. Arguments, kernels, results (bitwise)
 * and errors are those of hs_k_attn_decode. The split partials live in a
 * static device array of HS_K_ATTN_DECODE_NOALLOC_MAX_FLOATS floats
 * (32 MiB), one per GPU, held until the process ends; a call needing more,
 * B * n_heads * ceil(max_ctx / 128) * (head_dim + 2) floats, returns
 * HS_ERANGE before touching the GPU. Every call on one GPU uses the same
 * array, so calls that overlap in time on one GPU (other streams, other
 * threads) race and give wrong results: order them. */
#define HS_K_ATTN_DECODE_NOALLOC_MAX_FLOATS (8ll * 1024 * 1024)
hs_status hs_k_attn_decode_noalloc(const void* q, int64_t ldq, const void* pool,
                                   const int32_t* block_table, const int32_t* ctx, void* out,
                                   int64_t ldo, int32_t B, int32_t n_heads, int32_t n_kv_heads,
                                   int32_t head_dim, int32_t max_blocks, int32_t max_ctx,
                                   void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HS_KERNEL_H */
