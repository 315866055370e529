// Single-kernel entry points (include/hs_kernel.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>
#include <utility>
#include <vector>

#include "../../include/hs_kernel.h"
#include "hs_host.h"
#include "hs_kernels.h"
#include "kernel_entry.h"

using namespace hs;

namespace {
// Split-k workspace of hs_k_gemm, one per device, allocated on first use and
// kept until the process ends (calls on one device must not overlap).
struct GemmWs {
  float* part = nullptr;
  uint32_t* flags = nullptr;
};
constexpr int64_t kWsPartFloats = 2ll * 256 * 256 * 256;  // 2 slots x 256 workgroups x 256x256
constexpr int64_t kWsFlags = 1 << 16;

hs_status gemm_ws(GemmWs** out) {
  static GemmWs ws[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
    return fail(HS_EHIP, "hipGetDevice failed");
  GemmWs& w = ws[dev];
  if (!w.part) {
    float* p = nullptr;
    uint32_t* f = nullptr;
    if (hipMalloc(&p, kWsPartFloats * sizeof(float)) != hipSuccess) return fail(HS_ENOMEM, "gemm workspace");
    if (hipMalloc(&f, kWsFlags * sizeof(uint32_t)) != hipSuccess ||
        hipMemset(f, 0, kWsFlags * sizeof(uint32_t)) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess) {
      (void)hipFree(p);
      if (f) (void)hipFree(f);
      return fail(HS_ENOMEM, "gemm workspace");
    }
    w.part = p;
    w.flags = f;
  }
  *out = &w;
  return HS_OK;
}

hs_status launched(hipError_t e, const char* what) {
  if (e == hipErrorInvalidValue) return fail(HS_EINVAL, std::string(what) + ": unsupported shape");
  if (e != hipSuccess) return fail(HS_EHIP, std::string(what) + ": " + hipGetErrorString(e));
  return HS_OK;
}
}  // namespace

hs_status gemm_call(GemmArgs a, int32_t epi, void* stream) {
  GemmWs* ws = nullptr;
  const hs_status r = gemm_ws(&ws);
  if (r != HS_OK) return r;
  a.part = ws->part;
  a.part_floats = kWsPartFloats;
  a.flags = ws->flags;
  a.flags_n = kWsFlags;
  return launched(gemm(a, epi, static_cast<hipStream_t>(stream), nullptr), "gemm");
}

extern "C" hs_status hs_k_gemm(const void* X, int64_t ldx, const void* Wt, void* Y, int64_t ldy,
                               const void* R, int64_t ldr, int32_t M, int32_t N, int32_t K,
                               int32_t epi, void* stream) {
  try {
    if (!X || !Wt || !Y) return fail(HS_EINVAL, "null operand");
    GemmArgs a{static_cast<const bf16_t*>(X), ldx, static_cast<const bf16_t*>(Wt), Y, ldy,
               static_cast<const bf16_t*>(R), ldr, M, N, K};
    return gemm_call(a, epi, stream);
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}

extern "C" hs_status hs_k_gemm_rmsnorm(const void* X, int64_t ldx, const void* g, float eps,
                                       const void* Wt, void* Y, int64_t ldy, const void* R,
                                       int64_t ldr, int32_t M, int32_t N, int32_t K, int32_t epi,
                                       void* stream) {
  try {
    if (!X || !g || !Wt || !Y) return fail(HS_EINVAL, "null operand");
    if (M < 1 || M > 16 || K % 64) return fail(HS_EINVAL, "needs 1 <= M <= 16 and K % 64 == 0");
    GemmArgs a{static_cast<const bf16_t*>(X), ldx, static_cast<const bf16_t*>(Wt), Y, ldy,
               static_cast<const bf16_t*>(R), ldr, M, N, K};
    a.norm_gain = static_cast<const bf16_t*>(g);
    a.norm_eps = eps;
    return gemm_call(a, epi, stream);
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}

extern "C" hs_status hs_k_attn_prefill(const void* qkv, void* out, const int32_t* cu, int32_t n,
                                       int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                       void* stream) {
  try {
    if (!qkv || !out || !cu || n < 1) return fail(HS_EINVAL, "bad arguments");
    if (n_kv_heads < 1 || n_heads % n_kv_heads) return fail(HS_EINVAL, "bad head counts");
    if (cu[0] != 0) return fail(HS_EINVAL, "cu_seqlens[0] must be 0");
    std::vector<int32_t> tiles;
    int64_t tiles128 = 0;
    for (int i = 0; i < n; ++i) {
      const int len = cu[i + 1] - cu[i];
      if (len < 1) return fail(HS_EINVAL, "sequence lengths must be >= 1");
      tiles128 += (len + 127) / 128;
    }
    const int waves = attn_prefill_waves(tiles128, n_heads);
    for (int i = 0; i < n; ++i)
      for (int q = 0; q < cu[i + 1] - cu[i]; q += 16 * waves) {
        tiles.push_back(i);
        tiles.push_back(q);
      }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t* d = nullptr;
    const size_t nb = (size_t)(n + 1 + tiles.size()) * 4;
    if (hipMalloc(reinterpret_cast<void**>(&d), nb) != hipSuccess)
      return fail(HS_ENOMEM, "device allocation failed");
    hipError_t e = hipMemcpy(d, cu, (n + 1) * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(d + n + 1, tiles.data(), tiles.size() * 4, hipMemcpyHostToDevice);
    const int ld = (n_heads + 2 * n_kv_heads) * head_dim;
    AttnPrefillArgs a{static_cast<const bf16_t*>(qkv), ld, static_cast<bf16_t*>(out),
                      n_heads * head_dim, d, d + n + 1, (int)(tiles.size() / 2), n_heads,
                      n_kv_heads, head_dim, waves, 16 * waves, 0.0};
    if (e == hipSuccess) e = attn_prefill(a, s, nullptr);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipFree(d);
    return launched(e, "attn_prefill");
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}

namespace {
// Split partials of hs_k_attn_decode, one buffer per device, grown on demand.
struct DecodeWs {
  float* buf = nullptr;
  int64_t floats = 0;
};
}  // namespace

int64_t hs::attn_decode_ws_floats(int32_t B, int32_t n_heads, int32_t head_dim, int32_t max_ctx) {
  if (B < 1 || n_heads < 1 || head_dim < 1 || max_ctx < 1) return 0;
  const int64_t max_splits = (max_ctx + kDecodeSplit - 1) / kDecodeSplit;
  return (int64_t)B * n_heads * max_splits * (head_dim + 2);
}

hs_status hs::attn_decode_check(const void* q, const void* pool, const int32_t* block_table,
                            const int32_t* ctx, const void* out, bool rope, const float* cos_t,
                            const float* sin_t, int32_t max_pos, int32_t B, int32_t n_heads,
                            int32_t n_kv_heads, int32_t max_blocks, int32_t max_ctx) {
  if (!q || !pool || !block_table || !ctx || !out || B < 1 || max_ctx < 1)
    return fail(HS_EINVAL, "bad arguments");
  if (n_kv_heads < 1 || n_heads < 1 || n_heads % n_kv_heads)
    return fail(HS_EINVAL, "bad head counts");
  if (max_blocks < (max_ctx + 15) / 16) return fail(HS_EINVAL, "block table too narrow");
  if (rope && (!cos_t || !sin_t || max_pos < max_ctx))
    return fail(HS_EINVAL, "RoPE tables missing or shorter than max_ctx");
  return HS_OK;
}

hs_status hs::attn_decode_run(const void* q, int64_t ldq, const void* pool, bf16_t* pool_w,
                          const int32_t* block_table, const int32_t* ctx, const float* cos_t,
                          const float* sin_t, int32_t max_pos, void* out, int64_t ldo, int32_t B,
                          int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                          int32_t max_blocks, int32_t max_ctx, float* ws, void* stream) {
  const int max_splits = (max_ctx + kDecodeSplit - 1) / kDecodeSplit;
  AttnDecodeArgs a{static_cast<const bf16_t*>(q), ldq, static_cast<const bf16_t*>(pool),
                   block_table, ctx, ws, ws + (int64_t)B * n_heads * max_splits * head_dim,
                   static_cast<bf16_t*>(out), ldo, B, n_heads, n_kv_heads, head_dim, max_blocks,
                   max_splits, max_splits, 0.0};
  a.pool_w = pool_w;
  a.cos_t = cos_t;
  a.sin_t = sin_t;
  a.max_pos = max_pos;
  return launched(attn_decode(a, static_cast<hipStream_t>(stream), nullptr), "attn_decode");
}

namespace {
hs_status attn_decode_entry(const void* q, int64_t ldq, const void* pool, bf16_t* pool_w,
                            const int32_t* block_table, const int32_t* ctx, const float* cos_t,
                            const float* sin_t, int32_t max_pos, void* out, int64_t ldo,
                            int32_t B, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                            int32_t max_blocks, int32_t max_ctx, void* stream) {
  const hs_status chk = attn_decode_check(q, pool, block_table, ctx, out, pool_w != nullptr,
                                          cos_t, sin_t, max_pos, B, n_heads, n_kv_heads,
                                          max_blocks, max_ctx);
  if (chk != HS_OK) return chk;
  static DecodeWs ws[64];
  int dev = 0;
  const hipError_t ge = hipGetDevice(&dev);
  if (ge != hipSuccess || dev < 0 || dev >= 64)
    return fail(HS_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(ge));
  const int64_t need = attn_decode_ws_floats(B, n_heads, head_dim, max_ctx);
  DecodeWs& w = ws[dev];
  if (w.floats < need) {
    if (w.buf) {
      (void)hipDeviceSynchronize();
      (void)hipFree(w.buf);
      w.buf = nullptr;
      w.floats = 0;
    }
    if (hipMalloc(reinterpret_cast<void**>(&w.buf), need * sizeof(float)) != hipSuccess)
      return fail(HS_ENOMEM, "attention workspace");
    w.floats = need;
  }
  return attn_decode_run(q, ldq, pool, pool_w, block_table, ctx, cos_t, sin_t, max_pos, out, ldo,
                         B, n_heads, n_kv_heads, head_dim, max_blocks, max_ctx, w.buf, stream);
}
}  // namespace

extern "C" hs_status hs_k_attn_decode(const void* q, int64_t ldq, const void* pool,
                                      const int32_t* block_table, const int32_t* ctx, void* out,
                                      int64_t ldo, int32_t B, int32_t n_heads, int32_t n_kv_heads,
                                      int32_t head_dim, int32_t max_blocks, int32_t max_ctx,
                                      void* stream) {
  try {
    return attn_decode_entry(q, ldq, pool, nullptr, block_table, ctx, nullptr, nullptr, 0, out,
                             ldo, B, n_heads, n_kv_heads, head_dim, max_blocks, max_ctx, stream);
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}

extern "C" hs_status hs_k_attn_decode_rope(const void* qkv, int64_t ldqkv, void* pool,
                                           const int32_t* block_table, const int32_t* ctx,
                                           const float* cos_t, const float* sin_t,
                                           int32_t max_pos, void* out, int64_t ldo, int32_t B,
                                           int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                           int32_t max_blocks, int32_t max_ctx, void* stream) {
  try {
    if (!pool) return fail(HS_EINVAL, "bad arguments");
    if (ldqkv < (int64_t)(n_heads + 2 * n_kv_heads) * head_dim)
      return fail(HS_EINVAL, "qkv rows narrower than the query, key and value heads");
    return attn_decode_entry(qkv, ldqkv, pool, static_cast<bf16_t*>(pool), block_table, ctx,
                             cos_t, sin_t, max_pos, out, ldo, B, n_heads, n_kv_heads, head_dim,
                             max_blocks, max_ctx, stream);
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}

extern "C" hs_status hs_k_argmax(const float* logits, int32_t n_rows, int32_t n_cols,
                                 int32_t* out, void* stream) {
  try {
    if (!logits || !out || n_rows < 1 || n_cols < 1 || n_cols % 4)
      return fail(HS_EINVAL, "needs logits, out, n_rows >= 1 and n_cols % 4 == 0");
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t* part = nullptr;
    const size_t nb = (size_t)n_rows * argmax_chunks(n_cols) * 2 * sizeof(int32_t);
    if (hipMalloc(reinterpret_cast<void**>(&part), nb) != hipSuccess)
      return fail(HS_ENOMEM, "device allocation failed");
    hipError_t e = argmax_rows(logits, n_rows, n_cols, part, out, s, nullptr);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipFree(part);
    return launched(e, "argmax");
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}

extern "C" hs_status hs_k_rmsnorm(const void* x, const void* g, void* out, int32_t rows,
                                  int32_t hidden, float eps, void* stream) {
  try {
    if (!x || !g || !out || rows < 1) return fail(HS_EINVAL, "bad arguments");
    return launched(rmsnorm(static_cast<const bf16_t*>(x), hidden, nullptr, rows, hidden,
                            static_cast<const bf16_t*>(g), eps, static_cast<bf16_t*>(out), hidden,
                            static_cast<hipStream_t>(stream), nullptr),
                    "rmsnorm");
  } catch (...) {
    return fail(HS_EINVAL, "unexpected internal error");
  }
}
