// Decode attention with its split partials in a static device array
// (hs_k_attn_decode_noalloc in include/hs_kernel.h): for callers that cannot
// allocate device memory. The kernels are those of hs_k_attn_decode.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/hs_kernel.h"
#include "hs_host.h"
#include "kernel_entry.h"

namespace {

// 32 MiB of split partials per device. Every call on a device shares it and
// it keeps the last call's contents: the split kernel writes every partial
// the merge kernel uses before the merge reads it, so nothing needs clearing.
constexpr int64_t kScratchFloats = HS_K_ATTN_DECODE_NOALLOC_MAX_FLOATS;
static __device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
float* g_ptr[kMaxDevices] = {};  // device address of `scratch` on each device

// The device address of this device's copy of `scratch`, looked up with the
// device current on the first call that runs there. In host code the name
// `scratch` is only a handle for the symbol lookup, never an address.
hs_status scratch_ptr(float** out) {
  int dev = 0;
  const hipError_t ge = hipGetDevice(&dev);
  if (ge != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return hs::fail(HS_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(ge));
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return hs::fail(HS_EHIP, std::string("hipGetSymbolAddress(scratch): ") +
                                   hipGetErrorString(e));
    g_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_ptr[dev];
  return HS_OK;
}

}  // namespace

extern "C" hs_status hs_k_attn_decode_noalloc(const void* q, int64_t ldq, const void* pool,
                                              const int32_t* block_table, const int32_t* ctx,
                                              void* out, int64_t ldo, int32_t B, int32_t n_heads,
                                              int32_t n_kv_heads, int32_t head_dim,
                                              int32_t max_blocks, int32_t max_ctx, void* stream) {
  try {
    const hs_status chk =
        hs::attn_decode_check(q, pool, block_table, ctx, out, false, nullptr, nullptr, 0, B,
                              n_heads, n_kv_heads, max_blocks, max_ctx);
    if (chk != HS_OK) return chk;
    const int64_t need = hs::attn_decode_ws_floats(B, n_heads, head_dim, max_ctx);
    if (need > kScratchFloats)
      return hs::fail(HS_ERANGE, "B * n_heads * ceil(max_ctx / 128) * (head_dim + 2) = " +
                                     std::to_string(need) + " floats exceeds the static " +
                                     "workspace of " + std::to_string(kScratchFloats));
    float* ws = nullptr;
    const hs_status r = scratch_ptr(&ws);
    if (r != HS_OK) return r;
    return hs::attn_decode_run(q, ldq, pool, nullptr, block_table, ctx, nullptr, nullptr, 0, out,
                               ldo, B, n_heads, n_kv_heads, head_dim, max_blocks, max_ctx, ws,
                               stream);
  } catch (...) {
    return hs::fail(HS_EINVAL, "unexpected internal error");
  }
}
