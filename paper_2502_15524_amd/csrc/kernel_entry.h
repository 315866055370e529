// Shared pieces of the decode-attention entry points (hs_k_attn_decode,
// hs_k_attn_decode_rope and the variant with a static workspace): argument
// checks, the size of the split-partials workspace and the launch itself.
#pragma once

#include <stdint.h>

#include "../../include/hs.h"

namespace hs {

typedef uint16_t bf16_t;

// Floats of split partials a decode-attention launch needs: per sequence and
// query head, one [head_dim] output and one (max, sum) pair per 128-token
// split of max_ctx. 0 for non-positive sizes.
int64_t attn_decode_ws_floats(int32_t B, int32_t n_heads, int32_t head_dim, int32_t max_ctx);

// HS_OK or HS_EINVAL (with the message set) for the host-visible argument
// rules of hs_k_attn_decode; `rope` adds the rules of the RoPE form.
hs_status attn_decode_check(const void* q, const void* pool, const int32_t* block_table,
                            const int32_t* ctx, const void* out, bool rope, const float* cos_t,
                            const float* sin_t, int32_t max_pos, int32_t B, int32_t n_heads,
                            int32_t n_kv_heads, int32_t max_blocks, int32_t max_ctx);

// Enqueues the split and merge kernels on `stream` with the partials in `ws`
// (at least attn_decode_ws_floats(...) floats of device memory). pool_w set
// selects the form with the step's RoPE and cache append folded in.
hs_status attn_decode_run(const void* q, int64_t ldq, const void* pool, bf16_t* pool_w,
                          const int32_t* block_table, const int32_t* ctx, const float* cos_t,
                          const float* sin_t, int32_t max_pos, void* out, int64_t ldo, int32_t B,
                          int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                          int32_t max_blocks, int32_t max_ctx, float* ws, void* stream);

}  // namespace hs
