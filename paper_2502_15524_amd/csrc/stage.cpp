// The stage engine behind the C ABI: device weight image with per-chunk
// upload events, paged KV pools with a host-side block manager, the prefill
// and decode layer loops, and KV export / import / merge.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <set>
#include <string>
#include <vector>

#include "../../include/hs.h"
#include "hs_host.h"
#include "hs_kernels.h"

using namespace hs;

namespace {

std::string hip_msg(const char* what, hipError_t e) {
  return std::string(what) + ": " + hipGetErrorString(e);
}

#define HIPTRY(expr)                                              \
  do {                                                            \
    hipError_t _e = (expr);                                       \
    if (_e != hipSuccess) return fail(HS_EHIP, hip_msg(#expr, _e)); \
  } while (0)

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

struct Seq {
  int32_t n_tokens = 0;
  std::vector<int32_t> blocks;
  int32_t kv_begin = 0, kv_end = 0;  // layers whose cache this stage holds for it
};

struct Chunk {
  uint64_t off, bytes;
  hipEvent_t ev;
  bool done;
};

struct Pending {
  std::string name, site;
  hipEvent_t a, b;
  double flops, bytes;
};

struct Stat {
  std::string name, site;
  int64_t launches = 0;
  double ms = 0, flops = 0, bytes = 0;
};

constexpr int kRing = 4;
constexpr int kBlock = 16;

uint64_t al(uint64_t x) { return align_up(x, 256); }

}  // namespace

struct hs_stage {
  hs_model_cfg cfg{};
  int32_t begin = 0, end = 0;  // serving range
  int32_t rb = 0, re = 0;      // resident range
  hs_stage_opts opts{};
  int device = 0;
  ImageLayout L;
  uint8_t* d_image = nullptr;

  // KV pools: [resident layer][block][2][n_kv][16][D]
  uint8_t* d_kv = nullptr;
  uint64_t unit_bytes = 0, layer_pool_bytes = 0;
  int32_t num_blocks = 0, max_blocks_per_seq = 0;
  std::vector<int32_t> free_blocks;  // stack; back() is handed out next
  std::map<int64_t, Seq> seqs;

  std::vector<hipStream_t> copy;
  int next_copy = 0;
  // Completion of the latest call: the event its end recorded (own_done, or
  // the metadata slot's event of a call that used one: one event record per
  // call, each costing a fence on the stream).
  hipEvent_t own_done = nullptr;
  hipEvent_t last_done = nullptr;
  bool last_valid = false;
  int cur_meta = -1;      // metadata slot of the call in progress
  bool cur_desc = false;  // the call in progress pulled copy descriptors

  std::map<uint64_t, Chunk> chunks;
  std::vector<char> layer_landed;
  bool embed_landed = false, head_landed = false;

  // workspace
  uint8_t* d_ws = nullptr;
  bf16_t *w_x = nullptr, *w_u = nullptr, *w_qkv = nullptr, *w_attn = nullptr, *w_act = nullptr,
         *w_last = nullptr;
  float *w_logits = nullptr, *w_part_o = nullptr, *w_part_ml = nullptr;
  int32_t* w_argmax = nullptr;    // per-chunk partial results of the greedy argmax
  float* w_gpart = nullptr;       // split-k partial tiles of the projection GEMMs
  uint32_t* w_gflags = nullptr;   // their per-tile arrival counters (kept at zero)
  int64_t gpart_floats = 0, gflags_n = 0;
  float *d_cos = nullptr, *d_sin = nullptr;
  int32_t max_splits = 0;
  int64_t ws_rows = 0;

  // per-call metadata ring (pinned host -> device)
  uint8_t* h_meta[kRing] = {};
  uint8_t* d_meta[kRing] = {};
  hipEvent_t meta_ev[kRing] = {};
  bool meta_used[kRing] = {};
  int meta_next = 0;
  uint64_t meta_bytes = 0;

  // KV copy descriptors (grown on demand)
  uint8_t* h_desc = nullptr;
  uint8_t* d_desc = nullptr;
  uint64_t desc_cap = 0;
  hipEvent_t desc_ev = nullptr;
  bool desc_used = false;

  // host-staged KV migration: device staging blob and the chunk copies of
  // the last transfer (offset, bytes, completion event)
  uint8_t* d_stage = nullptr;
  uint64_t stage_cap = 0;
  struct Xfer {
    uint64_t off, bytes;
    hipEvent_t ev;
    bool done;
  };
  std::vector<Xfer> xfer;

  bool timing = false;
  std::string timing_sites;  // ",site,site@layer," or empty for every site
  int cur_layer = -1;        // decoder layer being enqueued (-1: none)
  std::vector<Pending> pending;
  std::map<std::string, Stat> stats;
  std::vector<hipEvent_t> ev_pool;

  ~hs_stage();
};

hs_stage::~hs_stage() {
  DeviceGuard g(device);
  for (auto s : copy) (void)hipStreamSynchronize(s);
  if (last_valid) (void)hipEventSynchronize(last_done);
  for (auto& kv : chunks) (void)hipEventDestroy(kv.second.ev);
  for (auto& p : pending) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  for (auto e : ev_pool) (void)hipEventDestroy(e);
  for (int i = 0; i < kRing; ++i) {
    if (meta_ev[i]) (void)hipEventDestroy(meta_ev[i]);
    if (h_meta[i]) (void)hipHostFree(h_meta[i]);
    if (d_meta[i]) (void)hipFree(d_meta[i]);
  }
  if (desc_ev) (void)hipEventDestroy(desc_ev);
  if (h_desc) (void)hipHostFree(h_desc);
  if (d_desc) (void)hipFree(d_desc);
  if (own_done) (void)hipEventDestroy(own_done);
  for (auto s : copy) (void)hipStreamDestroy(s);
  for (auto& x : xfer) (void)hipEventDestroy(x.ev);
  if (d_stage) (void)hipFree(d_stage);
  if (d_ws) (void)hipFree(d_ws);
  if (d_cos) (void)hipFree(d_cos);
  if (d_sin) (void)hipFree(d_sin);
  if (d_kv) (void)hipFree(d_kv);
  if (d_image) (void)hipFree(d_image);
}

namespace {

// ------------------------------------------------------------------ helpers

// Work goes on the caller's stream; NULL is the null stream.
hipStream_t pick(hs_stage*, void* stream) { return static_cast<hipStream_t>(stream); }

// Every call waits for the previous one, so calls on different streams stay
// ordered (on the same stream the wait costs nothing measurable).
hs_status begin_call(hs_stage* st, hipStream_t s) {
  if (st->last_valid) HIPTRY(hipStreamWaitEvent(s, st->last_done, 0));
  return HS_OK;
}

// Record the call's completion; a call that pulled metadata or copy
// descriptors records the event that guards that buffer's reuse, which then
// also orders the next call.
hs_status end_call(hs_stage* st, hipStream_t s) {
  hipEvent_t e = st->cur_meta >= 0 ? st->meta_ev[st->cur_meta]
                 : st->cur_desc     ? st->desc_ev
                                    : st->own_done;
  st->cur_meta = -1;
  st->cur_desc = false;
  HIPTRY(hipEventRecord(e, s));
  st->last_done = e;
  st->last_valid = true;
  return HS_OK;
}

// Ends a call that pulled metadata on every path: an error return after the
// pull still records the slot's event, so the host never rewrites a slot that
// a queued pull may read.
struct CallEnd {
  hs_stage* st;
  hipStream_t s;
  bool armed = true;
  ~CallEnd() {
    if (armed) (void)end_call(st, s);
  }
  hs_status finish() {
    armed = false;
    return end_call(st, s);
  }
};

hipEvent_t pool_event(hs_stage* st) {
  if (!st->ev_pool.empty()) {
    hipEvent_t e = st->ev_pool.back();
    st->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Projection GEMM arguments with the stage's split-k workspace attached.
GemmArgs gemm_args(const hs_stage* st, const bf16_t* X, int64_t ldx, const bf16_t* W, void* Y,
                   int64_t ldy, const bf16_t* R, int64_t ldr, int M, int N, int K) {
  GemmArgs g{X, ldx, W, Y, ldy, R, ldr, M, N, K};
  g.part = st->w_gpart;
  g.part_floats = st->gpart_floats;
  g.flags = st->w_gflags;
  g.flags_n = st->gflags_n;
  return g;
}

// Launch through a kernel launcher, bracketed by events when timing is on
// for this call site.
bool timed_site(const hs_stage* st, const char* site) {
  if (!st->timing) return false;
  if (st->timing_sites.empty()) return true;
  const std::string key = std::string(",") + site + ",";
  if (st->timing_sites.find(key) != std::string::npos) return true;
  if (st->cur_layer < 0) return false;
  const std::string one = std::string(",") + site + "@" + std::to_string(st->cur_layer) + ",";
  return st->timing_sites.find(one) != std::string::npos;
}

template <typename F>
hs_status run(hs_stage* st, hipStream_t s, const char* site, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  const bool timed = timed_site(st, site);
  if (timed) {
    a = pool_event(st);
    b = pool_event(st);
    if (!a || !b) return fail(HS_EHIP, "event creation failed");
    HIPTRY(hipEventRecord(a, s));
  }
  LaunchInfo info{"", 0, 0};
  hipError_t e = launch(&info);
  if (e != hipSuccess) return fail(HS_EHIP, hip_msg(info.name && *info.name ? info.name : "kernel launch", e));
  if (timed) {
    HIPTRY(hipEventRecord(b, s));
    st->pending.push_back(Pending{info.name ? info.name : "?", site, a, b, info.flops, info.bytes});
  }
  return HS_OK;
}

// Metadata slot for one call: host pinned + device, sized meta_bytes.
struct Meta {
  int slot;
  int32_t* h;
  int32_t* d;
  uint64_t used = 0;  // int32 elements
  uint64_t cap = 0;
  bool overflow = false;
  // Reserve n int32 values (64-aligned); returns the host and device views.
  int32_t* take(uint64_t n, int32_t** dptr) {
    static thread_local std::vector<int32_t> sink;
    const uint64_t off = used, sz = (n + 63) / 64 * 64;
    if (off + sz > cap) {  // sizes are bounded at creation; never expected
      overflow = true;
      sink.assign(sz, 0);
      *dptr = d;
      return sink.data();
    }
    used += sz;
    *dptr = d + off;
    return h + off;
  }
};

hs_status meta_acquire(hs_stage* st, Meta* m) {
  const int i = st->meta_next;
  st->meta_next = (i + 1) % kRing;
  if (st->meta_used[i]) HIPTRY(hipEventSynchronize(st->meta_ev[i]));
  m->slot = i;
  m->h = reinterpret_cast<int32_t*>(st->h_meta[i]);
  m->d = reinterpret_cast<int32_t*>(st->d_meta[i]);
  m->used = 0;
  m->cap = st->meta_bytes / 4;
  m->overflow = false;
  return HS_OK;
}

// Pull the call's metadata into device memory; the slot's event is recorded
// when the call ends (end_call).
hs_status meta_upload(hs_stage* st, const Meta& m, hipStream_t s) {
  if (m.overflow || m.used * 4 > st->meta_bytes) return fail(HS_EINVAL, "internal: metadata overflow");
  st->cur_meta = m.slot;
  st->meta_used[m.slot] = true;
  const hipError_t e = meta_pull(m.h, m.d, (int64_t)m.used, s);
  if (e != hipSuccess) return fail(HS_EHIP, hip_msg("metadata pull", e));
  return HS_OK;
}

// Is [b, e) covered by submitted chunks? Appends the events still pending.
bool covered(hs_stage* st, uint64_t b, uint64_t e, std::vector<hipEvent_t>* evs, bool* all_done) {
  bool done = true;
  auto it = st->chunks.upper_bound(b);
  if (it != st->chunks.begin()) {
    auto p = std::prev(it);
    if (p->second.off + p->second.bytes > b) it = p;
  }
  uint64_t pos = b;
  while (pos < e) {
    if (it == st->chunks.end() || it->second.off > pos) return false;
    Chunk& c = it->second;
    if (!c.done) {
      if (hipEventQuery(c.ev) == hipSuccess)
        c.done = true;
      else {
        done = false;
        if (evs) evs->push_back(c.ev);
      }
    }
    pos = c.off + c.bytes;
    ++it;
  }
  if (all_done) *all_done = done;
  return true;
}

struct Need {
  uint64_t b, e;
  char* landed;
  std::vector<hipEvent_t> evs;
};

// Readiness of the weights a forward pass over the serving range needs.
hs_status gather_needs(hs_stage* st, std::vector<Need>* embed, std::vector<Need>* layers,
                       std::vector<Need>* head) {
  auto one = [&](uint64_t b, uint64_t e, char* landed, const char* what, int l,
                 std::vector<Need>* out) -> hs_status {
    Need n{b, e, landed, {}};
    if (!*landed) {
      bool done = false;
      if (!covered(st, b, e, &n.evs, &done)) {
        std::string m = std::string("weights of ") + what;
        if (l >= 0) m += " " + std::to_string(l);
        return fail(HS_ENOTREADY, m + " were not submitted with hs_stage_load_chunk");
      }
      if (done) *landed = 1;
    }
    out->push_back(std::move(n));
    return HS_OK;
  };
  static char dummy;
  (void)dummy;
  if (st->begin == 0) {
    hs_status r = one(st->L.embed, st->L.embed_end, reinterpret_cast<char*>(&st->embed_landed),
                      "the embedding", -1, embed);
    if (r != HS_OK) return r;
  }
  for (int l = st->begin; l < st->end; ++l) {
    const LayerSlots& s = st->L.layers[l - st->rb];
    hs_status r = one(s.begin, s.end, &st->layer_landed[l - st->rb], "layer", l, layers);
    if (r != HS_OK) return r;
  }
  if (st->end == st->cfg.n_layers) {
    hs_status r = one(st->L.head_begin, st->L.head_end, reinterpret_cast<char*>(&st->head_landed),
                      "the LM head", -1, head);
    if (r != HS_OK) return r;
  }
  return HS_OK;
}

hs_status wait_need(hipStream_t s, const Need& n) {
  for (hipEvent_t e : n.evs) HIPTRY(hipStreamWaitEvent(s, e, 0));
  return HS_OK;
}

const bf16_t* W(const hs_stage* st, uint64_t off) {
  return reinterpret_cast<const bf16_t*>(st->d_image + off);
}

bf16_t* pool(const hs_stage* st, int layer) {
  return reinterpret_cast<bf16_t*>(st->d_kv + (uint64_t)(layer - st->rb) * st->layer_pool_bytes);
}

int32_t blocks_for(int32_t n) { return (n + kBlock - 1) / kBlock; }

// One decoder layer on rows [0, T) of x (bf16 residual stream, in place).
// The stage's first layer reads its residual stream from xin (the caller's
// input, or x itself) and writes x, so an input in another buffer is never
// copied first.
struct LayerCall {
  bool decode;
  int T;
  const bf16_t* xin;
  const int32_t *pos, *slot;             // device
  const int32_t *cu, *tiles;             // prefill
  int n_tiles, attn_waves;
  double attn_flops;
  const int32_t *bt, *ctx;               // decode
  int call_splits;
  double kv_read_bytes;
};

hs_status layer_forward_(hs_stage* st, int l, bf16_t* x, const LayerCall& c, hipStream_t s);

// One decoder layer, with the layer recorded for layer-qualified timing sites.
hs_status layer_forward(hs_stage* st, int l, bf16_t* x, const LayerCall& c, hipStream_t s) {
  st->cur_layer = l;
  const hs_status r = layer_forward_(st, l, x, c, s);
  st->cur_layer = -1;
  return r;
}

hs_status layer_forward_(hs_stage* st, int l, bf16_t* x, const LayerCall& c, hipStream_t s) {
  const hs_model_cfg& m = st->cfg;
  const LayerSlots& ls = st->L.layers[l - st->rb];
  const int H = m.hidden, D = m.head_dim, F = m.ffn;
  const int FA = (int)round64(F);  // activation row stride: zero columns up to a multiple of 64
  const int NQKV = (m.n_heads + 2 * m.n_kv_heads) * D, QD = m.n_heads * D;
  // Up to 16 tokens (decode batches) the skinny GEMMs apply the two norms
  // themselves and read the residual stream directly.
  const bool fuse_norm = c.T <= 16;
  const bf16_t* xr = l == st->begin ? c.xin : x;  // residual stream before the o projection
  hs_status r;
  if (!fuse_norm) {
    r = run(st, s, "attn_norm", [&](LaunchInfo* i) {
      return rmsnorm(xr, H, nullptr, c.T, H, W(st, ls.attn_norm), m.rms_eps, st->w_u, H, s, i);
    });
    if (r != HS_OK) return r;
  }
  r = run(st, s, "qkv", [&](LaunchInfo* i) {
    GemmArgs g = fuse_norm
                     ? gemm_args(st, xr, H, W(st, ls.qkv), st->w_qkv, NQKV, nullptr, 0, c.T, NQKV, H)
                     : gemm_args(st, st->w_u, H, W(st, ls.qkv), st->w_qkv, NQKV, nullptr, 0, c.T, NQKV, H);
    if (fuse_norm) g.norm_gain = W(st, ls.attn_norm), g.norm_eps = m.rms_eps;
    // the image stores q and k heads with their RoPE halves interleaved
    g.rope_q_cols = QD;
    g.rope_kv_cols = m.n_kv_heads * D;
    g.rope_d = D;
    if (c.decode) return gemm(g, EPI_STORE, s, i);  // the attention kernel rotates and appends
    g.rope_pos = c.pos;
    g.rope_slot = c.slot;
    g.rope_cos = st->d_cos;
    g.rope_sin = st->d_sin;
    g.rope_max_pos = st->opts.max_ctx;
    g.rope_pool = pool(st, l);
    return gemm(g, EPI_QKV_ROPE, s, i);
  });
  if (r != HS_OK) return r;
  if (!c.decode) {
    r = run(st, s, "attn", [&](LaunchInfo* i) {
      AttnPrefillArgs a{st->w_qkv, NQKV, st->w_attn, QD, c.cu, c.tiles, c.n_tiles,
                        m.n_heads, m.n_kv_heads, D, c.attn_waves, 16 * c.attn_waves,
                        c.attn_flops};
      return attn_prefill(a, s, i);
    });
  } else {
    r = run(st, s, "attn", [&](LaunchInfo* i) {
      AttnDecodeArgs a{st->w_qkv, NQKV, pool(st, l), c.bt, c.ctx, st->w_part_o, st->w_part_ml,
                       st->w_attn, QD, c.T, m.n_heads, m.n_kv_heads, D, st->max_blocks_per_seq,
                       st->max_splits, c.call_splits, c.kv_read_bytes};
      a.pool_w = pool(st, l);
      a.cos_t = st->d_cos;
      a.sin_t = st->d_sin;
      a.max_pos = st->opts.max_ctx;
      return attn_decode(a, s, i);
    });
  }
  if (r != HS_OK) return r;
  r = run(st, s, "o_proj", [&](LaunchInfo* i) {
    GemmArgs g = gemm_args(st, st->w_attn, QD, W(st, ls.o), x, H, xr, H, c.T, H, QD);
    return gemm(g, EPI_RESID, s, i);
  });
  if (r != HS_OK) return r;
  if (!fuse_norm) {
    r = run(st, s, "ffn_norm", [&](LaunchInfo* i) {
      return rmsnorm(x, H, nullptr, c.T, H, W(st, ls.ffn_norm), m.rms_eps, st->w_u, H, s, i);
    });
    if (r != HS_OK) return r;
  }
  r = run(st, s, "gate_up", [&](LaunchInfo* i) {
    GemmArgs g = fuse_norm
                     ? gemm_args(st, x, H, W(st, ls.gateup), st->w_act, FA, nullptr, 0, c.T, 2 * F, H)
                     : gemm_args(st, st->w_u, H, W(st, ls.gateup), st->w_act, FA, nullptr, 0, c.T, 2 * F, H);
    if (fuse_norm) g.norm_gain = W(st, ls.ffn_norm), g.norm_eps = m.rms_eps;
    return gemm(g, EPI_SWIGLU, s, i);
  });
  if (r != HS_OK) return r;
  return run(st, s, "down", [&](LaunchInfo* i) {
    GemmArgs g = gemm_args(st, st->w_act, FA, W(st, ls.down), x, H, x, H, c.T, H, F);
    return gemm(g, EPI_RESID, s, i);
  });
}

// Final norm on the given rows, LM head (fp32 logits), greedy argmax.
hs_status head_forward(hs_stage* st, const bf16_t* x, const int32_t* rows, int n, float* logits,
                       int32_t* out, hipStream_t s) {
  const hs_model_cfg& m = st->cfg;
  const int H = m.hidden;
  hs_status r = run(st, s, "final_norm", [&](LaunchInfo* i) {
    return rmsnorm(x, H, rows, n, H, W(st, st->L.final_norm), m.rms_eps, st->w_last, H, s, i);
  });
  if (r != HS_OK) return r;
  float* lg = logits ? logits : st->w_logits;
  r = run(st, s, "lm_head", [&](LaunchInfo* i) {
    GemmArgs g = gemm_args(st, st->w_last, H, W(st, st->L.lm_head), lg, m.vocab, nullptr, 0, n, m.vocab, H);
    return gemm(g, EPI_F32, s, i);
  });
  if (r != HS_OK) return r;
  return run(st, s, "argmax", [&](LaunchInfo* i) {
    return argmax_rows(lg, n, m.vocab, st->w_argmax, out, s, i);
  });
}

bool is_device_ptr(const void* p) {
  if (!p) return false;
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice;
}

bool is_pinned_host_ptr(const void* p) {
  if (!p) return false;
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

// Grow the KV-copy descriptor buffers to hold n units.
hs_status desc_reserve(hs_stage* st, uint64_t n) {
  const uint64_t need = al(n * 8) * 2 + al(n * 4);
  if (st->desc_used) HIPTRY(hipEventSynchronize(st->desc_ev));
  if (need <= st->desc_cap) return HS_OK;
  if (st->h_desc) HIPTRY(hipHostFree(st->h_desc));
  if (st->d_desc) HIPTRY(hipFree(st->d_desc));
  st->h_desc = nullptr;
  st->d_desc = nullptr;
  st->desc_cap = 0;
  const uint64_t cap = std::max<uint64_t>(need, 1 << 16);
  if (hipHostMalloc(reinterpret_cast<void**>(&st->h_desc), cap, hipHostMallocCoherent) != hipSuccess)
    return fail(HS_ENOMEM, "pinned descriptor buffer allocation failed");
  if (hipMalloc(reinterpret_cast<void**>(&st->d_desc), cap) != hipSuccess)
    return fail(HS_ENOMEM, "device descriptor buffer allocation failed");
  st->desc_cap = cap;
  return HS_OK;
}

struct Units {
  std::vector<uint64_t> src, dst;
  std::vector<int32_t> valid;
};

// Pull the descriptors (the first desc_bytes of the pinned buffer) into the
// device descriptor buffer and the blob header, if any, straight into the
// blob, with one kernel (a copy command costs a stream fence of its own).
// Header sizes are multiples of 16 bytes (64 + 16 per sequence record).
hs_status pull_desc(hs_stage* st, const uint8_t* h, uint64_t desc_bytes,
                    const std::vector<uint8_t>* head, void* head_dst, hipStream_t s) {
  const uint64_t hn = head ? head->size() : 0;
  if (hn % 16) return fail(HS_EINVAL, "internal: blob header not a multiple of 16 bytes");
  const hipError_t e = meta_pull(
      reinterpret_cast<const int32_t*>(h), reinterpret_cast<int32_t*>(st->d_desc),
      (int64_t)(desc_bytes / 4), s, reinterpret_cast<const int32_t*>(h + desc_bytes),
      static_cast<int32_t*>(head_dst), (int64_t)(hn / 4));
  if (e != hipSuccess) return fail(HS_EHIP, hip_msg("descriptor pull", e));
  return HS_OK;
}

// Upload descriptors (and optionally a blob header, copied to head_dst in the
// same upload) and launch the KV copy kernel on stream s. The descriptor
// buffer's guard event is recorded by the call's end_call (one upload per
// call).
hs_status copy_units(hs_stage* st, const Units& u, int zero_tail, hipStream_t s,
                     const std::vector<uint8_t>* head = nullptr, void* head_dst = nullptr) {
  const uint64_t n = u.src.size();
  const uint64_t hb = head ? al(head->size()) : 0;
  if (n == 0 && !head) return HS_OK;
  hs_status r = desc_reserve(st, n + hb / 8 + 1);
  if (r != HS_OK) return r;
  uint8_t* h = st->h_desc;
  const uint64_t o_dst = al(n * 8), o_val = 2 * al(n * 8), o_head = o_val + al(n * 4);
  memcpy(h, u.src.data(), n * 8);
  memcpy(h + o_dst, u.dst.data(), n * 8);
  memcpy(h + o_val, u.valid.data(), n * 4);
  if (head) memcpy(h + o_head, head->data(), head->size());
  r = pull_desc(st, h, o_head, head, head_dst, s);
  if (r != HS_OK) return r;
  st->cur_desc = true;  // the pull is queued: the call's end guards the buffer
  st->desc_used = true;
  const uint64_t* dsrc = reinterpret_cast<const uint64_t*>(st->d_desc);
  const uint64_t* ddst = reinterpret_cast<const uint64_t*>(st->d_desc + o_dst);
  const int32_t* dval = reinterpret_cast<const int32_t*>(st->d_desc + o_val);
  if (n > 0) {
    r = run(st, s, "kv_copy", [&](LaunchInfo* i) {
      return kv_copy(dsrc, ddst, dval, (int)n, (int64_t)st->unit_bytes, st->cfg.head_dim,
                     zero_tail, s, i);
    });
    if (r != HS_OK) return r;
  }
  return HS_OK;
}

// Upload the descriptors of `u` (and a blob header to head_dst) on stream s
// without launching; returns the device views.
hs_status desc_upload(hs_stage* st, const Units& u, hipStream_t s, const std::vector<uint8_t>* head,
                      void* head_dst, const uint64_t** dsrc, const uint64_t** ddst,
                      const int32_t** dval) {
  const uint64_t n = u.src.size();
  const uint64_t hb = head ? al(head->size()) : 0;
  hs_status r = desc_reserve(st, n + hb / 8 + 1);
  if (r != HS_OK) return r;
  uint8_t* h = st->h_desc;
  const uint64_t o_dst = al(n * 8), o_val = 2 * al(n * 8), o_head = o_val + al(n * 4);
  memcpy(h, u.src.data(), n * 8);
  memcpy(h + o_dst, u.dst.data(), n * 8);
  memcpy(h + o_val, u.valid.data(), n * 4);
  if (head) memcpy(h + o_head, head->data(), head->size());
  r = pull_desc(st, h, o_head, head, head_dst, s);
  if (r != HS_OK) return r;
  *dsrc = reinterpret_cast<const uint64_t*>(st->d_desc);
  *ddst = reinterpret_cast<const uint64_t*>(st->d_desc + o_dst);
  *dval = reinterpret_cast<const int32_t*>(st->d_desc + o_val);
  return HS_OK;
}

// Grow the device staging blob of host-staged migration. Growing waits for
// the stage's queued work (the old buffer may still be in use).
hs_status stage_buffer(hs_stage* st, uint64_t bytes) {
  if (bytes <= st->stage_cap) return HS_OK;
  if (st->last_valid) HIPTRY(hipEventSynchronize(st->last_done));
  for (auto c : st->copy) HIPTRY(hipStreamSynchronize(c));
  if (st->d_stage) HIPTRY(hipFree(st->d_stage));
  st->d_stage = nullptr;
  st->stage_cap = 0;
  if (hipMalloc(reinterpret_cast<void**>(&st->d_stage), bytes) != hipSuccess)
    return fail(HS_ENOMEM, "KV staging buffer allocation failed");
  st->stage_cap = bytes;
  return HS_OK;
}

// Forget the previous transfer's chunk events (the stage's ordering already
// covers them: every transfer joins its copy streams into the call stream).
void xfer_reset(hs_stage* st) {
  for (auto& x : st->xfer) (void)hipEventDestroy(x.ev);
  st->xfer.clear();
}

// The sequence table and free-block list an import works on: the stage's
// own, or copies when several blobs are validated before any of them counts.
typedef std::map<int64_t, Seq> SeqTable;

// Validate a blob header held in host memory against the stage's geometry
// and the given sequence table. Changes nothing; import_commit then
// registers the sequences.
hs_status import_check(const hs_stage* st, const SeqTable& seqs, size_t n_free,
                       const uint8_t* head, uint64_t head_len, uint64_t bytes,
                       BlobHeader* hout, std::vector<BlobRecord>* rout) {
  BlobHeader h;
  std::vector<BlobRecord> recs;
  hs_status r = blob_decode_head(head, head_len, &h, &recs);
  if (r != HS_OK) return r;
  if (h.total_bytes != bytes) return fail(HS_EINVAL, "blob length does not match its header");
  if (h.n_kv_heads != st->cfg.n_kv_heads || h.head_dim != st->cfg.head_dim ||
      h.block_size != kBlock)
    return fail(HS_EINVAL, "blob KV geometry differs from the stage's");
  if (h.layer_begin < st->rb || h.layer_end > st->re)
    return fail(HS_EINVAL, "blob layers are not resident in this stage");
  int64_t need_blocks = 0, new_seqs = 0;
  for (const BlobRecord& rc : recs) {
    if (rc.n_tokens > st->opts.max_ctx) return fail(HS_EINVAL, "blob sequence longer than max_ctx");
    auto it = seqs.find(rc.seq_id);
    if (it == seqs.end()) {
      need_blocks += rc.n_blocks;
      ++new_seqs;
    } else {
      const Seq& q = it->second;
      if (q.n_tokens != rc.n_tokens)
        return fail(HS_EINVAL, "blob token count differs from the live sequence's");
      if (!(h.layer_end == q.kv_begin || h.layer_begin == q.kv_end ||
            (h.layer_begin >= q.kv_begin && h.layer_end <= q.kv_end)))
        return fail(HS_EINVAL, "blob layers are not adjacent to the sequence's cached layers");
    }
  }
  if ((int64_t)seqs.size() + new_seqs > st->opts.max_seqs)
    return fail(HS_ENOMEM, "no free sequence slots");
  if (need_blocks > (int64_t)n_free) return fail(HS_ENOMEM, "not enough free KV blocks");
  *hout = h;
  *rout = std::move(recs);
  return HS_OK;
}

// Units one import of this blob copies (layers x blocks of every record).
uint64_t import_unit_count(const BlobHeader& h, const std::vector<BlobRecord>& recs) {
  uint64_t blocks = 0;
  for (const BlobRecord& rc : recs) blocks += (uint64_t)rc.n_blocks;
  return (uint64_t)(h.layer_end - h.layer_begin) * blocks;
}

// Register the blob's sequences (new ones get fresh blocks) after
// import_check accepted it; cannot fail.
void import_commit(SeqTable& seqs, std::vector<int32_t>& free_blocks, const BlobHeader& h,
                   const std::vector<BlobRecord>& recs) {
  for (const BlobRecord& rc : recs) {
    auto it = seqs.find(rc.seq_id);
    if (it == seqs.end()) {
      Seq q;
      q.n_tokens = rc.n_tokens;
      q.kv_begin = h.layer_begin;
      q.kv_end = h.layer_end;
      for (int b = 0; b < rc.n_blocks; ++b) {
        q.blocks.push_back(free_blocks.back());
        free_blocks.pop_back();
      }
      seqs.emplace(rc.seq_id, std::move(q));
    } else {
      Seq& q = it->second;
      q.kv_begin = std::min(q.kv_begin, h.layer_begin);
      q.kv_end = std::max(q.kv_end, h.layer_end);
    }
  }
}

// Units of an import: blob payload (at base) -> the stage's pools.
void import_units(const hs_stage* st, const SeqTable& seqs, const BlobHeader& h,
                  const std::vector<BlobRecord>& recs, uint64_t base, Units* out) {
  Units& u = *out;
  uint64_t unit = 0;
  for (int l = h.layer_begin; l < h.layer_end; ++l)
    for (const BlobRecord& rc : recs) {
      const Seq& q = seqs.at(rc.seq_id);
      for (int b = 0; b < rc.n_blocks; ++b, ++unit) {
        u.src.push_back(base + h.payload_offset + unit * st->unit_bytes);
        u.dst.push_back((uint64_t)(uintptr_t)pool(st, l) + (uint64_t)q.blocks[b] * st->unit_bytes);
        u.valid.push_back(kBlock);
      }
    }
}

bool same_model(const hs_model_cfg& a, const hs_model_cfg& b) {
  return a.n_layers == b.n_layers && a.hidden == b.hidden && a.n_heads == b.n_heads &&
         a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim && a.ffn == b.ffn &&
         a.vocab == b.vocab && a.rms_eps == b.rms_eps && a.rope_base == b.rope_base;
}

}  // namespace

// =================================================================== C ABI

#define ABI_BEGIN try {
#define ABI_END                                                   \
  }                                                               \
  catch (const std::bad_alloc&) {                                 \
    return fail(HS_ENOMEM, "host allocation failed");             \
  }                                                               \
  catch (...) {                                                   \
    return fail(HS_EINVAL, "unexpected internal error");          \
  }

extern "C" hs_status hs_stage_create(const hs_model_cfg* cfg, int32_t layer_begin,
                                     int32_t layer_end, const hs_stage_opts* opts, int32_t device,
                                     hs_stage** out) {
  ABI_BEGIN
  if (!out) return fail(HS_EINVAL, "null output handle");
  *out = nullptr;
  std::string why;
  if (!cfg_valid(cfg, &why)) return fail(HS_EINVAL, why);
  if (!opts) return fail(HS_EINVAL, "null options");
  const hs_model_cfg& m = *cfg;
  if (layer_begin < 0 || layer_end > m.n_layers || layer_begin > layer_end)
    return fail(HS_EINVAL, "serving range must satisfy 0 <= begin <= end <= n_layers");
  int32_t rb = opts->resident_begin, re = opts->resident_end;
  if (re == 0 && rb == 0) {
    rb = layer_begin;
    re = layer_end;
  }
  if (rb < 0 || re > m.n_layers || rb >= re)
    return fail(HS_EINVAL, "resident range must be a non-empty part of the model");
  if (layer_begin != layer_end && (layer_begin < rb || layer_end > re))
    return fail(HS_EINVAL, "serving range must lie inside the resident range");
  if (opts->max_seqs < 1 || opts->max_ctx < 1 || opts->max_batch_tokens < 1)
    return fail(HS_EINVAL, "max_seqs, max_ctx and max_batch_tokens must be >= 1");
  if (opts->kv_block_size != kBlock) return fail(HS_EINVAL, "kv_block_size must be 16");
  if (opts->kv_num_blocks < 0) return fail(HS_EINVAL, "kv_num_blocks must be >= 0");
  if (opts->n_copy_streams < 1 || opts->n_copy_streams > 8)
    return fail(HS_EINVAL, "n_copy_streams must be in 1..8");
  int n_dev = 0;
  HIPTRY(hipGetDeviceCount(&n_dev));
  if (device < 0 || device >= n_dev) return fail(HS_EINVAL, "no such HIP device");
  DeviceGuard dg(device);

  hs_stage* st = new hs_stage();
  auto bail = [&](hs_status r) {
    delete st;
    return r;
  };
  st->cfg = m;
  st->begin = layer_begin;
  st->end = layer_end;
  st->rb = rb;
  st->re = re;
  st->opts = *opts;
  st->opts.resident_begin = rb;
  st->opts.resident_end = re;
  st->device = device;
  hs_status r = build_layout(m, rb, re, &st->L);
  if (r != HS_OK) return bail(r);
  st->layer_landed.assign(re - rb, 0);

  const int D = m.head_dim, H = m.hidden, F = m.ffn, V = m.vocab;
  const int NQKV = (m.n_heads + 2 * m.n_kv_heads) * D, QD = m.n_heads * D;
  st->max_blocks_per_seq = blocks_for(opts->max_ctx);
  st->num_blocks = opts->kv_num_blocks ? opts->kv_num_blocks
                                       : opts->max_seqs * st->max_blocks_per_seq;
  st->unit_bytes = blob_unit_bytes(m.n_kv_heads, D, kBlock);
  st->layer_pool_bytes = (uint64_t)st->num_blocks * st->unit_bytes;
  st->max_splits = (opts->max_ctx + kDecodeSplit - 1) / kDecodeSplit;
  st->ws_rows = std::max(opts->max_batch_tokens, opts->max_seqs);

  if (hipMalloc(reinterpret_cast<void**>(&st->d_image), st->L.bytes) != hipSuccess)
    return bail(fail(HS_ENOMEM, "device weight image allocation failed"));
  if (hipMalloc(reinterpret_cast<void**>(&st->d_kv), st->layer_pool_bytes * (re - rb)) != hipSuccess)
    return bail(fail(HS_ENOMEM, "KV pool allocation failed"));

  // activation workspace
  const uint64_t R = (uint64_t)st->ws_rows, S = (uint64_t)opts->max_seqs;
  uint64_t off = 0;
  std::vector<uint64_t> offs;
  // split-k workspace: two 256 x 128 fp32 partial tiles per CU, a counter
  // per 128 x 64 output tile of the widest projection
  int cus = 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
      cus <= 0)
    cus = 256;
  const int64_t max_n = std::max<int64_t>(std::max(NQKV, 2 * F), std::max(H, V));
  st->gpart_floats = R > 64 ? 2ll * cus * 256 * 128 : 0;
  st->gflags_n = R > 64 ? ((max_n + 127) / 128) * (int64_t)((R + 63) / 64) : 0;
  for (uint64_t sz : {R * H * 2, R * H * 2, R * NQKV * 2, R * QD * 2, R * round64(F) * 2, S * H * 2,
                      S * V * 4, S * m.n_heads * st->max_splits * (uint64_t)D * 4,
                      S * m.n_heads * st->max_splits * 2 * 4, (uint64_t)st->gpart_floats * 4,
                      (uint64_t)st->gflags_n * 4, S * (uint64_t)argmax_chunks(V) * 8}) {
    offs.push_back(off);
    off = al(off + sz);
  }
  if (hipMalloc(reinterpret_cast<void**>(&st->d_ws), off) != hipSuccess)
    return bail(fail(HS_ENOMEM, "workspace allocation failed"));
  // zero once: padding columns of the activations stay zero for good
  if (hipMemset(st->d_ws, 0, off) != hipSuccess || hipDeviceSynchronize() != hipSuccess)
    return bail(fail(HS_EHIP, "workspace initialisation failed"));
  st->w_x = reinterpret_cast<bf16_t*>(st->d_ws + offs[0]);
  st->w_u = reinterpret_cast<bf16_t*>(st->d_ws + offs[1]);
  st->w_qkv = reinterpret_cast<bf16_t*>(st->d_ws + offs[2]);
  st->w_attn = reinterpret_cast<bf16_t*>(st->d_ws + offs[3]);
  st->w_act = reinterpret_cast<bf16_t*>(st->d_ws + offs[4]);
  st->w_last = reinterpret_cast<bf16_t*>(st->d_ws + offs[5]);
  st->w_logits = reinterpret_cast<float*>(st->d_ws + offs[6]);
  st->w_part_o = reinterpret_cast<float*>(st->d_ws + offs[7]);
  st->w_part_ml = reinterpret_cast<float*>(st->d_ws + offs[8]);
  st->w_gpart = st->gpart_floats ? reinterpret_cast<float*>(st->d_ws + offs[9]) : nullptr;
  st->w_gflags = st->gflags_n ? reinterpret_cast<uint32_t*>(st->d_ws + offs[10]) : nullptr;
  st->w_argmax = reinterpret_cast<int32_t*>(st->d_ws + offs[11]);

  // RoPE table: angle pos * base^(-2i/D) in double, stored as float.
  {
    const int half = D / 2;
    std::vector<float> c((size_t)opts->max_ctx * half), sn((size_t)opts->max_ctx * half);
    for (int p = 0; p < opts->max_ctx; ++p)
      for (int i = 0; i < half; ++i) {
        const double ang = (double)p * pow((double)m.rope_base, -2.0 * i / D);
        c[(size_t)p * half + i] = (float)cos(ang);
        sn[(size_t)p * half + i] = (float)sin(ang);
      }
    if (hipMalloc(reinterpret_cast<void**>(&st->d_cos), c.size() * 4) != hipSuccess ||
        hipMalloc(reinterpret_cast<void**>(&st->d_sin), sn.size() * 4) != hipSuccess)
      return bail(fail(HS_ENOMEM, "RoPE table allocation failed"));
    if (hipMemcpy(st->d_cos, c.data(), c.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(st->d_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
      return bail(fail(HS_EHIP, "RoPE table upload failed"));
  }

  // streams (the weight-upload streams only: compute runs on the caller's
  // stream), events
  for (int i = 0; i < opts->n_copy_streams; ++i) {
    hipStream_t s = nullptr;
    if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess)
      return bail(fail(HS_EHIP, "stream creation failed"));
    st->copy.push_back(s);
  }
  if (hipEventCreateWithFlags(&st->own_done, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&st->desc_ev, hipEventDisableTiming) != hipSuccess)
    return bail(fail(HS_EHIP, "event creation failed"));

  // metadata ring
  {
    const uint64_t T = opts->max_batch_tokens, MB = st->max_blocks_per_seq;
    const uint64_t pre = 2 * T + (S + 1) + 2 * (T / 64 + S + 1) + S;
    const uint64_t dec = 3 * S + S * MB;
    st->meta_bytes = ((std::max(pre, dec) + 64 * 8) * 4 + 4095) / 4096 * 4096;
    for (int i = 0; i < kRing; ++i) {
      if (hipHostMalloc(reinterpret_cast<void**>(&st->h_meta[i]), st->meta_bytes,
                        hipHostMallocCoherent) != hipSuccess ||
          hipMalloc(reinterpret_cast<void**>(&st->d_meta[i]), st->meta_bytes) != hipSuccess)
        return bail(fail(HS_ENOMEM, "metadata buffer allocation failed"));
      if (hipEventCreateWithFlags(&st->meta_ev[i], hipEventDisableTiming) != hipSuccess)
        return bail(fail(HS_EHIP, "event creation failed"));
    }
  }

  st->free_blocks.reserve(st->num_blocks);
  for (int32_t b = st->num_blocks - 1; b >= 0; --b) st->free_blocks.push_back(b);
  *out = st;
  clear_error();
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_destroy(hs_stage* st) {
  ABI_BEGIN
  delete st;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_sync(hs_stage* st) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  DeviceGuard dg(st->device);
  if (st->last_valid) HIPTRY(hipEventSynchronize(st->last_done));
  for (auto s : st->copy) HIPTRY(hipStreamSynchronize(s));
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_load_chunk(hs_stage* st, uint64_t off, const void* src,
                                         uint64_t bytes) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  if (!src) return fail(HS_EINVAL, "null source");
  if (bytes == 0) return fail(HS_EINVAL, "empty chunk");
  if (off > st->L.bytes || bytes > st->L.bytes - off)
    return fail(HS_EINVAL, "chunk lies outside the weight image");
  auto it = st->chunks.lower_bound(off);
  if (it != st->chunks.end() && it->second.off < off + bytes)
    return fail(HS_EINVAL, "chunk overlaps a chunk already submitted");
  if (it != st->chunks.begin()) {
    auto p = std::prev(it);
    if (p->second.off + p->second.bytes > off)
      return fail(HS_EINVAL, "chunk overlaps a chunk already submitted");
  }
  DeviceGuard dg(st->device);
  hipStream_t s = st->copy[st->next_copy];
  hipEvent_t ev = nullptr;
  HIPTRY(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
  hipError_t e = hipMemcpyAsync(st->d_image + off, src, bytes, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipEventRecord(ev, s);
  if (e != hipSuccess) {
    (void)hipEventDestroy(ev);
    return fail(HS_EHIP, hip_msg("weight chunk copy", e));
  }
  st->next_copy = (st->next_copy + 1) % (int)st->copy.size();
  st->chunks.emplace(off, Chunk{off, bytes, ev, false});
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_loaded(hs_stage* st, int32_t* layers_ready, uint64_t* watermark) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  DeviceGuard dg(st->device);
  uint64_t pos = 0;
  for (auto& kv : st->chunks) {
    Chunk& c = kv.second;
    if (!c.done && hipEventQuery(c.ev) == hipSuccess) c.done = true;
    if (c.off != pos || !c.done) break;
    pos = c.off + c.bytes;
  }
  int32_t n = 0;
  for (int l = st->rb; l < st->re; ++l) {
    const LayerSlots& s = st->L.layers[l - st->rb];
    bool done = false;
    if (!covered(st, s.begin, s.end, nullptr, &done) || !done) break;
    ++n;
  }
  if (layers_ready) *layers_ready = n;
  if (watermark) *watermark = pos;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_invalidate_weights(hs_stage* st) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  hs_status r = hs_stage_sync(st);
  if (r != HS_OK) return r;
  DeviceGuard dg(st->device);
  for (auto& kv : st->chunks) HIPTRY(hipEventDestroy(kv.second.ev));
  st->chunks.clear();
  std::fill(st->layer_landed.begin(), st->layer_landed.end(), 0);
  st->embed_landed = st->head_landed = false;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_prefill(hs_stage* st, int32_t n, const int64_t* ids,
                                      const int32_t* lens, const void* in, void* out,
                                      float* logits_opt, void* stream) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  if (st->begin == st->end) return fail(HS_ESTATE, "stage has an empty serving range");
  if (n < 1 || !ids || !lens || !in || !out) return fail(HS_EINVAL, "bad prefill arguments");
  const bool first = st->begin == 0, last = st->end == st->cfg.n_layers;
  if (logits_opt && !last) return fail(HS_EINVAL, "logits are only produced by the last stage");
  int64_t T = 0;
  int64_t need_blocks = 0;
  std::set<int64_t> uniq;
  for (int i = 0; i < n; ++i) {
    if (lens[i] < 1) return fail(HS_EINVAL, "prompt lengths must be >= 1");
    if (lens[i] > st->opts.max_ctx) return fail(HS_EINVAL, "prompt longer than max_ctx");
    if (st->seqs.count(ids[i])) return fail(HS_EINVAL, "sequence id is already live");
    if (!uniq.insert(ids[i]).second) return fail(HS_EINVAL, "repeated sequence id");
    T += lens[i];
    need_blocks += blocks_for(lens[i]);
  }
  if (T > st->opts.max_batch_tokens) return fail(HS_EINVAL, "more tokens than max_batch_tokens");
  if ((int64_t)st->seqs.size() + n > st->opts.max_seqs)
    return fail(HS_ENOMEM, "no free sequence slots");
  if (need_blocks > (int64_t)st->free_blocks.size()) return fail(HS_ENOMEM, "not enough free KV blocks");
  DeviceGuard dg(st->device);
  std::vector<Need> ne, nl, nh;
  hs_status r = gather_needs(st, &ne, &nl, &nh);
  if (r != HS_OK) return r;

  hipStream_t s = pick(st, stream);
  Meta mt;
  r = meta_acquire(st, &mt);
  if (r != HS_OK) return r;
  // the new sequences and per-token metadata; the sequences take blocks from
  // the back of the free list (as popping would) but the stage's state only
  // changes once every launch has been enqueued, so a failed call leaves it
  // as it was
  int32_t *d_pos, *d_slot, *d_cu, *d_tiles, *d_last;
  int32_t* pos = mt.take(T, &d_pos);
  int32_t* slot = mt.take(T, &d_slot);
  int32_t* cu = mt.take(n + 1, &d_cu);
  std::vector<std::pair<int, int>> tiles;
  std::vector<Seq> fresh(n);
  size_t free_end = st->free_blocks.size();
  double attn_flops = 0;
  cu[0] = 0;
  for (int i = 0; i < n; ++i) {
    Seq& sq = fresh[i];
    sq.n_tokens = lens[i];
    sq.kv_begin = st->begin;
    sq.kv_end = st->end;
    for (int b = 0; b < blocks_for(lens[i]); ++b) sq.blocks.push_back(st->free_blocks[--free_end]);
    for (int p = 0; p < lens[i]; ++p) {
      pos[cu[i] + p] = p;
      slot[cu[i] + p] = sq.blocks[p / kBlock] * kBlock + p % kBlock;
    }
    cu[i + 1] = cu[i] + lens[i];
    attn_flops += 4.0 * st->cfg.n_heads * st->cfg.head_dim * 0.5 * (double)lens[i] * (lens[i] + 1);
  }
  // attention work tiles: q_tile queries of one sequence, longest rows first
  int64_t tiles128 = 0;
  for (int i = 0; i < n; ++i) tiles128 += (lens[i] + 127) / 128;
  const int attn_waves = attn_prefill_waves(tiles128, st->cfg.n_heads);
  const int q_tile = 16 * attn_waves;
  for (int i = 0; i < n; ++i)
    for (int q = 0; q < lens[i]; q += q_tile) tiles.emplace_back(i, q);
  std::stable_sort(tiles.begin(), tiles.end(),
                   [](const std::pair<int, int>& a, const std::pair<int, int>& b) {
                     return a.second > b.second;
                   });
  int32_t* tl = mt.take(2 * tiles.size(), &d_tiles);
  for (size_t i = 0; i < tiles.size(); ++i) {
    tl[2 * i] = tiles[i].first;
    tl[2 * i + 1] = tiles[i].second;
  }
  int32_t* lastr = mt.take(n, &d_last);
  for (int i = 0; i < n; ++i) lastr[i] = cu[i + 1] - 1;

  r = begin_call(st, s);
  if (r != HS_OK) return r;
  CallEnd ce{st, s};
  r = meta_upload(st, mt, s);
  if (r != HS_OK) return r;

  const int H = st->cfg.hidden;
  bf16_t* x = last ? st->w_x : static_cast<bf16_t*>(out);
  if (first) {
    r = wait_need(s, ne[0]);
    if (r != HS_OK) return r;
    r = run(st, s, "embed", [&](LaunchInfo* i) {
      return embed(static_cast<const int32_t*>(in), W(st, st->L.embed), st->cfg.vocab, H, (int)T,
                   x, s, i);
    });
    if (r != HS_OK) return r;
  }
  LayerCall c{};
  c.decode = false;
  c.T = (int)T;
  c.xin = first ? x : static_cast<const bf16_t*>(in);
  c.pos = d_pos;
  c.slot = d_slot;
  c.cu = d_cu;
  c.tiles = d_tiles;
  c.n_tiles = (int)tiles.size();
  c.attn_waves = attn_waves;
  c.attn_flops = attn_flops;
  for (int l = st->begin; l < st->end; ++l) {
    r = wait_need(s, nl[l - st->begin]);
    if (r != HS_OK) return r;
    r = layer_forward(st, l, x, c, s);
    if (r != HS_OK) return r;
  }
  if (last) {
    r = wait_need(s, nh[0]);
    if (r != HS_OK) return r;
    r = head_forward(st, x, d_last, n, logits_opt, static_cast<int32_t*>(out), s);
    if (r != HS_OK) return r;
  }
  st->free_blocks.resize(free_end);
  for (int i = 0; i < n; ++i) st->seqs.emplace(ids[i], std::move(fresh[i]));
  return ce.finish();
  ABI_END
}

extern "C" hs_status hs_stage_decode(hs_stage* st, int32_t n, const int64_t* ids, const void* in,
                                     void* out, float* logits_opt, void* stream) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  if (st->begin == st->end) return fail(HS_ESTATE, "stage has an empty serving range");
  if (n < 1 || !ids || !in || !out) return fail(HS_EINVAL, "bad decode arguments");
  if (n > st->ws_rows) return fail(HS_EINVAL, "more sequences than the workspace holds");
  const bool first = st->begin == 0, last = st->end == st->cfg.n_layers;
  if (logits_opt && !last) return fail(HS_EINVAL, "logits are only produced by the last stage");
  std::set<int64_t> uniq;
  int64_t need_blocks = 0;
  std::vector<Seq*> sq(n);
  for (int i = 0; i < n; ++i) {
    auto it = st->seqs.find(ids[i]);
    if (it == st->seqs.end()) return fail(HS_EINVAL, "unknown sequence id");
    if (!uniq.insert(ids[i]).second) return fail(HS_EINVAL, "repeated sequence id");
    Seq& q = it->second;
    if (q.kv_begin > st->begin || q.kv_end < st->end)
      return fail(HS_ESTATE, "sequence cache does not cover the serving layers");
    if (q.n_tokens + 1 > st->opts.max_ctx) return fail(HS_ERANGE, "sequence would exceed max_ctx");
    if (q.n_tokens % kBlock == 0) ++need_blocks;
    sq[i] = &q;
  }
  if (need_blocks > (int64_t)st->free_blocks.size()) return fail(HS_ENOMEM, "no free KV block");
  DeviceGuard dg(st->device);
  std::vector<Need> ne, nl, nh;
  hs_status r = gather_needs(st, &ne, &nl, &nh);
  if (r != HS_OK) return r;

  hipStream_t s = pick(st, stream);
  Meta mt;
  r = meta_acquire(st, &mt);
  if (r != HS_OK) return r;
  const int MB = st->max_blocks_per_seq;
  int32_t *d_pos, *d_slot, *d_ctx, *d_bt;
  int32_t* pos = mt.take(n, &d_pos);
  int32_t* slot = mt.take(n, &d_slot);
  int32_t* ctx = mt.take(n, &d_ctx);
  int32_t* bt = mt.take((uint64_t)n * MB, &d_bt);
  int call_splits = 1;
  double kv_bytes = 0;
  const double tok_bytes = 2.0 * st->cfg.n_kv_heads * st->cfg.head_dim * 2;
  // a sequence whose last block is full takes a new one from the back of the
  // free list; the stage's state changes only after the launches (see prefill)
  std::vector<int32_t> new_block(n, -1);
  size_t free_end = st->free_blocks.size();
  for (int i = 0; i < n; ++i) {
    const Seq& q = *sq[i];
    const int p = q.n_tokens;
    if (p % kBlock == 0) new_block[i] = st->free_blocks[--free_end];
    const int nb = (int)q.blocks.size() + (new_block[i] >= 0 ? 1 : 0);
    const int last_blk = new_block[i] >= 0 ? new_block[i] : q.blocks[p / kBlock];
    pos[i] = p;
    slot[i] = last_blk * kBlock + p % kBlock;
    ctx[i] = p + 1;
    for (int b = 0; b < MB; ++b)
      bt[(uint64_t)i * MB + b] = b < (int)q.blocks.size() ? q.blocks[b] : (b < nb ? new_block[i] : 0);
    call_splits = std::max(call_splits, (p + 1 + kDecodeSplit - 1) / kDecodeSplit);
    kv_bytes += (p + 1) * tok_bytes;
  }
  r = begin_call(st, s);
  if (r != HS_OK) return r;
  CallEnd ce{st, s};
  r = meta_upload(st, mt, s);
  if (r != HS_OK) return r;

  const int H = st->cfg.hidden;
  bf16_t* x = last ? st->w_x : static_cast<bf16_t*>(out);
  if (first) {
    r = wait_need(s, ne[0]);
    if (r != HS_OK) return r;
    r = run(st, s, "embed", [&](LaunchInfo* i) {
      return embed(static_cast<const int32_t*>(in), W(st, st->L.embed), st->cfg.vocab, H, n, x, s, i);
    });
    if (r != HS_OK) return r;
  }
  LayerCall c{};
  c.decode = true;
  c.T = n;
  c.xin = first ? x : static_cast<const bf16_t*>(in);
  c.pos = d_pos;
  c.slot = d_slot;
  c.bt = d_bt;
  c.ctx = d_ctx;
  c.call_splits = call_splits;
  c.kv_read_bytes = kv_bytes;

  for (int l = st->begin; l < st->end; ++l) {
    r = wait_need(s, nl[l - st->begin]);
    if (r != HS_OK) return r;
    r = layer_forward(st, l, x, c, s);
    if (r != HS_OK) return r;
  }
  if (last) {
    r = wait_need(s, nh[0]);
    if (r != HS_OK) return r;
    r = head_forward(st, x, nullptr, n, logits_opt, static_cast<int32_t*>(out), s);
    if (r != HS_OK) return r;
  }
  st->free_blocks.resize(free_end);
  for (int i = 0; i < n; ++i) {
    if (new_block[i] >= 0) sq[i]->blocks.push_back(new_block[i]);
    sq[i]->n_tokens += 1;
  }
  return ce.finish();
  ABI_END
}

extern "C" hs_status hs_seq_free(hs_stage* st, int64_t id) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  auto it = st->seqs.find(id);
  if (it == st->seqs.end()) return fail(HS_EINVAL, "unknown sequence id");
  // Blocks may still be read by enqueued work; later writers are ordered
  // after it because every call waits for the previous one.
  for (auto b = it->second.blocks.rbegin(); b != it->second.blocks.rend(); ++b)
    st->free_blocks.push_back(*b);
  st->seqs.erase(it);
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_seq_tokens(const hs_stage* st, int64_t id, int32_t* n_tokens) {
  ABI_BEGIN
  if (!st || !n_tokens) return fail(HS_EINVAL, "null argument");
  auto it = st->seqs.find(id);
  if (it == st->seqs.end()) return fail(HS_EINVAL, "unknown sequence id");
  *n_tokens = it->second.n_tokens;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_get_info(const hs_stage* st, hs_stage_info* o) {
  ABI_BEGIN
  if (!st || !o) return fail(HS_EINVAL, "null argument");
  o->layer_begin = st->begin;
  o->layer_end = st->end;
  o->resident_begin = st->rb;
  o->resident_end = st->re;
  o->live_seqs = (int32_t)st->seqs.size();
  o->free_blocks = (int32_t)st->free_blocks.size();
  o->total_blocks = st->num_blocks;
  o->block_size = kBlock;
  o->image_bytes = st->L.bytes;
  o->kv_bytes = st->layer_pool_bytes * (uint64_t)(st->re - st->rb);
  return HS_OK;
  ABI_END
}

// ---------------------------------------------------------------- KV blobs

namespace {

hs_status export_records(const hs_stage* st, int32_t n, const int64_t* ids,
                         std::vector<BlobRecord>* recs, BlobHeader* h) {
  if (st->begin == st->end) return fail(HS_ESTATE, "stage has an empty serving range");
  if (n < 0 || (n > 0 && !ids)) return fail(HS_EINVAL, "bad sequence list");
  std::set<int64_t> uniq;
  recs->clear();
  for (int i = 0; i < n; ++i) {
    auto it = st->seqs.find(ids[i]);
    if (it == st->seqs.end()) return fail(HS_EINVAL, "unknown sequence id");
    if (!uniq.insert(ids[i]).second) return fail(HS_EINVAL, "repeated sequence id");
    if (it->second.kv_begin > st->begin || it->second.kv_end < st->end)
      return fail(HS_ESTATE, "sequence cache does not cover the serving layers");
    recs->push_back(BlobRecord{ids[i], it->second.n_tokens, blocks_for(it->second.n_tokens)});
  }
  h->layer_begin = st->begin;
  h->layer_end = st->end;
  h->n_kv_heads = st->cfg.n_kv_heads;
  h->head_dim = st->cfg.head_dim;
  h->block_size = kBlock;
  blob_sizes(h, *recs);
  return HS_OK;
}

}  // namespace

extern "C" hs_status hs_kv_export_size(const hs_stage* st, int32_t n, const int64_t* ids,
                                       uint64_t* bytes) {
  ABI_BEGIN
  if (!st || !bytes) return fail(HS_EINVAL, "null argument");
  std::vector<BlobRecord> recs;
  BlobHeader h;
  hs_status r = export_records(st, n, ids, &recs, &h);
  if (r != HS_OK) return r;
  *bytes = h.total_bytes;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_kv_export(hs_stage* st, int32_t n, const int64_t* ids, void* dst,
                                  uint64_t cap, uint64_t* written, void* stream) {
  ABI_BEGIN
  if (!st || !written) return fail(HS_EINVAL, "null argument");
  std::vector<BlobRecord> recs;
  BlobHeader h;
  hs_status r = export_records(st, n, ids, &recs, &h);
  if (r != HS_OK) return r;
  *written = h.total_bytes;
  if (cap < h.total_bytes) return fail(HS_ERANGE, "destination smaller than the blob");
  DeviceGuard dg(st->device);
  if (!is_device_ptr(dst)) return fail(HS_EINVAL, "blob destination must be device memory");
  if ((uintptr_t)dst & 15) return fail(HS_EINVAL, "blob destination must be 16-byte aligned");
  std::vector<uint8_t> head = blob_encode_head(h, recs);
  Units u;
  uint64_t unit = 0;
  for (int l = st->begin; l < st->end; ++l)
    for (const BlobRecord& rc : recs) {
      const Seq& q = st->seqs.at(rc.seq_id);
      for (int b = 0; b < rc.n_blocks; ++b, ++unit) {
        u.src.push_back((uint64_t)(uintptr_t)pool(st, l) + (uint64_t)q.blocks[b] * st->unit_bytes);
        u.dst.push_back((uint64_t)(uintptr_t)dst + h.payload_offset + unit * st->unit_bytes);
        u.valid.push_back(std::min(kBlock, rc.n_tokens - b * kBlock));
      }
    }
  hipStream_t s = pick(st, stream);
  r = begin_call(st, s);
  if (r != HS_OK) return r;
  CallEnd ce{st, s};
  r = copy_units(st, u, 1, s, &head, dst);
  if (r != HS_OK) return r;
  return ce.finish();
  ABI_END
}

extern "C" hs_status hs_kv_import(hs_stage* st, const void* src, uint64_t bytes, void* stream) {
  ABI_BEGIN
  if (!st || !src) return fail(HS_EINVAL, "null argument");
  if (bytes < kBlobHeader) return fail(HS_EINVAL, "blob shorter than its header");
  DeviceGuard dg(st->device);
  if (!is_device_ptr(src)) return fail(HS_EINVAL, "blob source must be device memory");
  hipStream_t s = pick(st, stream);
  hs_status r = begin_call(st, s);
  if (r != HS_OK) return r;
  CallEnd ce{st, s};
  // one read covers the header and up to 256 sequence records; a blob with
  // more sequences takes a second read for the rest
  const uint64_t first = std::min<uint64_t>(bytes, kBlobHeader + kBlobRecord * 256);
  std::vector<uint8_t> head(first);
  HIPTRY(hipMemcpyAsync(head.data(), src, first, hipMemcpyDeviceToHost, s));
  HIPTRY(hipStreamSynchronize(s));
  int32_t ns = 0;
  memcpy(&ns, head.data() + 32, 4);
  if (ns < 0 || kBlobHeader + kBlobRecord * (uint64_t)ns > bytes)
    return fail(HS_EINVAL, "blob sequence count does not fit its length");
  const uint64_t need = kBlobHeader + kBlobRecord * (uint64_t)ns;
  if (need > first) {
    head.resize(need);
    HIPTRY(hipMemcpyAsync(head.data() + first, static_cast<const uint8_t*>(src) + first,
                          need - first, hipMemcpyDeviceToHost, s));
    HIPTRY(hipStreamSynchronize(s));
  } else {
    head.resize(need);
  }
  BlobHeader h;
  std::vector<BlobRecord> recs;
  r = import_check(st, st->seqs, st->free_blocks.size(), head.data(), head.size(), bytes, &h,
                   &recs);
  if (r != HS_OK) return r;
  r = desc_reserve(st, import_unit_count(h, recs) + 1);  // the last step that can fail
  if (r != HS_OK) return r;
  import_commit(st->seqs, st->free_blocks, h, recs);
  Units u;
  import_units(st, st->seqs, h, recs, (uint64_t)(uintptr_t)src, &u);
  r = copy_units(st, u, 0, s);
  if (r != HS_OK) return r;
  return ce.finish();
  ABI_END
}

extern "C" hs_status hs_kv_export_head(const hs_stage* st, int32_t n, const int64_t* ids,
                                       void* host_dst, uint64_t cap, uint64_t* written) {
  ABI_BEGIN
  if (!st || !written) return fail(HS_EINVAL, "null argument");
  std::vector<BlobRecord> recs;
  BlobHeader h;
  hs_status r = export_records(st, n, ids, &recs, &h);
  if (r != HS_OK) return r;
  std::vector<uint8_t> head = blob_encode_head(h, recs);
  *written = head.size();
  if (cap < head.size()) return fail(HS_ERANGE, "destination smaller than the blob head");
  if (!host_dst) return fail(HS_EINVAL, "null destination");
  memcpy(host_dst, head.data(), head.size());
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_kv_import_many(hs_stage* st, int32_t n_blobs, const void* const* srcs,
                                       const uint64_t* bytes, const void* const* heads,
                                       const uint64_t* head_bytes, void* stream) {
  ABI_BEGIN
  if (!st || n_blobs < 1 || !srcs || !bytes || !heads || !head_bytes)
    return fail(HS_EINVAL, "bad arguments");
  DeviceGuard dg(st->device);
  for (int i = 0; i < n_blobs; ++i) {
    if (!srcs[i] || !heads[i]) return fail(HS_EINVAL, "null blob or head");
    if (!is_device_ptr(srcs[i])) return fail(HS_EINVAL, "blob source must be device memory");
    if ((uintptr_t)srcs[i] & 15) return fail(HS_EINVAL, "blob source must be 16-byte aligned");
  }
  // every blob is checked against the state the blobs before it leave, on
  // copies of the sequence table and free list; the stage changes only once
  // all of them pass and the copy descriptors are reserved
  SeqTable seqs = st->seqs;
  std::vector<int32_t> free_blocks = st->free_blocks;
  std::vector<BlobHeader> hs_(n_blobs);
  std::vector<std::vector<BlobRecord>> recs(n_blobs);
  uint64_t units = 0;
  for (int i = 0; i < n_blobs; ++i) {
    hs_status r = import_check(st, seqs, free_blocks.size(),
                               static_cast<const uint8_t*>(heads[i]), head_bytes[i], bytes[i],
                               &hs_[i], &recs[i]);
    if (r != HS_OK) return fail(r, "blob " + std::to_string(i) + ": " + hs_last_error());
    import_commit(seqs, free_blocks, hs_[i], recs[i]);
    units += import_unit_count(hs_[i], recs[i]);
  }
  hs_status r = desc_reserve(st, units + 1);  // the last step that can fail
  if (r != HS_OK) return r;
  hipStream_t s = pick(st, stream);
  r = begin_call(st, s);
  if (r != HS_OK) return r;
  CallEnd ce{st, s};
  st->seqs.swap(seqs);
  st->free_blocks.swap(free_blocks);
  Units u;
  for (int i = 0; i < n_blobs; ++i)
    import_units(st, st->seqs, hs_[i], recs[i], (uint64_t)(uintptr_t)srcs[i], &u);
  r = copy_units(st, u, 0, s);
  if (r != HS_OK) return r;
  return ce.finish();
  ABI_END
}

// Host-staged migration: chunks are whole KV units; chunk j covers units
// [j * cu, (j + 1) * cu) (plus the header and records in the first chunk).
namespace {
struct ChunkPlan {
  uint64_t cu;        // units per chunk
  uint64_t n_chunks;
  uint64_t first, count;  // of chunk j, filled by at()
  uint64_t off, bytes;
};
ChunkPlan plan_chunks(const hs_stage* st, const BlobHeader& h, uint64_t units, uint64_t chunk_bytes) {
  ChunkPlan p{};
  p.cu = std::max<uint64_t>(1, chunk_bytes / st->unit_bytes);
  p.n_chunks = std::max<uint64_t>(1, (units + p.cu - 1) / p.cu);
  (void)h;
  return p;
}
void chunk_at(const hs_stage* st, const BlobHeader& h, uint64_t units, ChunkPlan* p, uint64_t j) {
  p->first = j * p->cu;
  p->count = std::min(p->cu, units - std::min(units, p->first));
  const uint64_t b0 = j == 0 ? 0 : h.payload_offset + p->first * st->unit_bytes;
  const uint64_t b1 = j + 1 == p->n_chunks ? h.total_bytes
                                           : h.payload_offset + (p->first + p->count) * st->unit_bytes;
  p->off = b0;
  p->bytes = b1 - b0;
}
}  // namespace

extern "C" hs_status hs_kv_export_host(hs_stage* st, int32_t n, const int64_t* ids, void* dst,
                                       uint64_t cap, uint64_t chunk_bytes, uint64_t* written,
                                       void* stream) {
  ABI_BEGIN
  if (!st || !written || !dst) return fail(HS_EINVAL, "null argument");
  if (chunk_bytes == 0) return fail(HS_EINVAL, "chunk_bytes must be positive");
  std::vector<BlobRecord> recs;
  BlobHeader h;
  hs_status r = export_records(st, n, ids, &recs, &h);
  if (r != HS_OK) return r;
  *written = h.total_bytes;
  if (cap < h.total_bytes) return fail(HS_ERANGE, "destination smaller than the blob");
  DeviceGuard dg(st->device);
  if (!is_pinned_host_ptr(dst)) return fail(HS_EINVAL, "blob destination must be pinned host memory");
  r = stage_buffer(st, h.total_bytes);
  if (r != HS_OK) return r;
  std::vector<uint8_t> head = blob_encode_head(h, recs);
  Units u;
  uint64_t unit = 0;
  for (int l = st->begin; l < st->end; ++l)
    for (const BlobRecord& rc : recs) {
      const Seq& q = st->seqs.at(rc.seq_id);
      for (int b = 0; b < rc.n_blocks; ++b, ++unit) {
        u.src.push_back((uint64_t)(uintptr_t)pool(st, l) + (uint64_t)q.blocks[b] * st->unit_bytes);
        u.dst.push_back((uint64_t)(uintptr_t)st->d_stage + h.payload_offset + unit * st->unit_bytes);
        u.valid.push_back(std::min(kBlock, rc.n_tokens - b * kBlock));
      }
    }
  hipStream_t s = pick(st, stream);
  r = begin_call(st, s);
  if (r != HS_OK) return r;
  xfer_reset(st);
  const uint64_t* dsrc;
  const uint64_t* ddst;
  const int32_t* dval;
  r = desc_upload(st, u, s, &head, st->d_stage, &dsrc, &ddst, &dval);
  if (r != HS_OK) return r;
  // Chunk j is gathered and then copied to the host on `stream` itself: the
  // copy of chunk j starts as soon as its gather ends, and the gather of
  // chunk j + 1 (a few microseconds against about a millisecond of copy per
  // 64 MiB) waits behind it. Copies on separate streams overlapped the
  // gathers but, with several exports queued back to back, the cross-stream
  // waits cut the host-link rate from 56 to 32-37 GB/s (MI355X).
  ChunkPlan p = plan_chunks(st, h, unit, chunk_bytes);
  for (uint64_t j = 0; j < p.n_chunks; ++j) {
    chunk_at(st, h, unit, &p, j);
    if (p.count > 0) {
      r = run(st, s, "kv_copy", [&](LaunchInfo* i) {
        return kv_copy(dsrc + p.first, ddst + p.first, dval + p.first, (int)p.count,
                       (int64_t)st->unit_bytes, st->cfg.head_dim, 1, s, i);
      });
      if (r != HS_OK) return r;
    }
    hipEvent_t landed = nullptr;
    HIPTRY(hipEventCreateWithFlags(&landed, hipEventDisableTiming));
    st->xfer.push_back({p.off, p.bytes, landed, false});
    HIPTRY(hipMemcpyAsync(static_cast<uint8_t*>(dst) + p.off, st->d_stage + p.off, p.bytes,
                          hipMemcpyDeviceToHost, s));
    HIPTRY(hipEventRecord(landed, s));
  }
  HIPTRY(hipEventRecord(st->desc_ev, s));
  st->desc_used = true;
  return end_call(st, s);
  ABI_END
}

extern "C" hs_status hs_kv_import_host(hs_stage* st, const void* src, uint64_t bytes,
                                       uint64_t chunk_bytes, void* stream) {
  ABI_BEGIN
  if (!st || !src) return fail(HS_EINVAL, "null argument");
  if (chunk_bytes == 0) return fail(HS_EINVAL, "chunk_bytes must be positive");
  if (bytes < kBlobHeader) return fail(HS_EINVAL, "blob shorter than its header");
  DeviceGuard dg(st->device);
  if (!is_pinned_host_ptr(src)) return fail(HS_EINVAL, "blob source must be pinned host memory");
  const uint8_t* hb = static_cast<const uint8_t*>(src);
  int32_t ns = 0;
  memcpy(&ns, hb + 32, 4);
  if (ns < 0 || kBlobHeader + kBlobRecord * (uint64_t)ns > bytes)
    return fail(HS_EINVAL, "blob sequence count does not fit its length");
  hipStream_t s = pick(st, stream);
  // the staging buffer must be free before the reservation changes state
  hs_status r = stage_buffer(st, bytes);
  if (r != HS_OK) return r;
  BlobHeader h;
  std::vector<BlobRecord> recs;
  r = import_check(st, st->seqs, st->free_blocks.size(), hb,
                   kBlobHeader + kBlobRecord * (uint64_t)ns, bytes, &h, &recs);
  if (r != HS_OK) return r;
  r = desc_reserve(st, import_unit_count(h, recs) + 1);  // the last step that can fail
  if (r != HS_OK) return r;
  import_commit(st->seqs, st->free_blocks, h, recs);
  Units u;
  import_units(st, st->seqs, h, recs, (uint64_t)(uintptr_t)st->d_stage, &u);
  r = begin_call(st, s);
  if (r != HS_OK) return r;
  xfer_reset(st);
  const uint64_t* dsrc;
  const uint64_t* ddst;
  const int32_t* dval;
  r = desc_upload(st, u, s, nullptr, nullptr, &dsrc, &ddst, &dval);
  if (r != HS_OK) return r;
  hipEvent_t ready = nullptr;  // earlier work on the staging buffer is done
  HIPTRY(hipEventCreateWithFlags(&ready, hipEventDisableTiming));
  HIPTRY(hipEventRecord(ready, s));
  for (auto c : st->copy) HIPTRY(hipStreamWaitEvent(c, ready, 0));
  HIPTRY(hipEventDestroy(ready));
  const uint64_t units = u.src.size();
  ChunkPlan p = plan_chunks(st, h, units, chunk_bytes);
  for (uint64_t j = 0; j < p.n_chunks; ++j) {
    chunk_at(st, h, units, &p, j);
    hipStream_t cs = st->copy[j % st->copy.size()];
    hipEvent_t landed = nullptr;
    HIPTRY(hipEventCreateWithFlags(&landed, hipEventDisableTiming));
    st->xfer.push_back({p.off, p.bytes, landed, false});
    HIPTRY(hipMemcpyAsync(st->d_stage + p.off, hb + p.off, p.bytes, hipMemcpyHostToDevice, cs));
    HIPTRY(hipEventRecord(landed, cs));
    // scatter this chunk's units as soon as it has landed
    HIPTRY(hipStreamWaitEvent(s, landed, 0));
    if (p.count > 0) {
      r = run(st, s, "kv_copy", [&](LaunchInfo* i) {
        return kv_copy(dsrc + p.first, ddst + p.first, dval + p.first, (int)p.count,
                       (int64_t)st->unit_bytes, st->cfg.head_dim, 0, s, i);
      });
      if (r != HS_OK) return r;
    }
  }
  HIPTRY(hipEventRecord(st->desc_ev, s));
  st->desc_used = true;
  return end_call(st, s);
  ABI_END
}

extern "C" hs_status hs_kv_host_progress(hs_stage* st, uint64_t* landed) {
  ABI_BEGIN
  if (!st || !landed) return fail(HS_EINVAL, "null argument");
  DeviceGuard dg(st->device);
  uint64_t pos = 0;
  for (auto& x : st->xfer) {
    if (!x.done && hipEventQuery(x.ev) == hipSuccess) x.done = true;
    if (x.off != pos || !x.done) break;
    pos = x.off + x.bytes;
  }
  *landed = pos;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_merge(hs_stage* dst, hs_stage* const* srcs, int32_t n_srcs,
                                    void* stream) {
  ABI_BEGIN
  if (!dst || (n_srcs > 0 && !srcs) || n_srcs < 1) return fail(HS_EINVAL, "bad merge arguments");
  std::set<const hs_stage*> uniq{dst};
  for (int i = 0; i < n_srcs; ++i) {
    if (!srcs[i]) return fail(HS_EINVAL, "null source stage");
    if (!uniq.insert(srcs[i]).second) return fail(HS_EINVAL, "a stage appears twice in the merge");
    if (!same_model(dst->cfg, srcs[i]->cfg)) return fail(HS_EINVAL, "stages of different models");
    if (srcs[i]->device != dst->device) return fail(HS_EINVAL, "stages on different devices");
    if (srcs[i]->begin == srcs[i]->end) return fail(HS_ESTATE, "source stage serves no layers");
  }
  // ranges: disjoint and contiguous, inside dst's resident range
  std::vector<std::pair<int, int>> rg;
  if (dst->begin != dst->end) rg.emplace_back(dst->begin, dst->end);
  for (int i = 0; i < n_srcs; ++i) rg.emplace_back(srcs[i]->begin, srcs[i]->end);
  std::sort(rg.begin(), rg.end());
  for (size_t i = 1; i < rg.size(); ++i)
    if (rg[i].first != rg[i - 1].second)
      return fail(HS_ESTATE, "serving ranges are not disjoint and contiguous");
  const int ub = rg.front().first, ue = rg.back().second;
  if (ub < dst->rb || ue > dst->re) return fail(HS_ESTATE, "union is not resident in the target");
  // live sets
  const auto& ref = srcs[0]->seqs;
  for (int i = 0; i < n_srcs; ++i) {
    const auto& ss = srcs[i]->seqs;
    if (ss.size() != ref.size()) return fail(HS_ESTATE, "sources hold different sequences");
    for (const auto& kv : ss) {
      auto it = ref.find(kv.first);
      if (it == ref.end() || it->second.n_tokens != kv.second.n_tokens)
        return fail(HS_ESTATE, "sources hold different sequences");
      if (kv.second.kv_begin > srcs[i]->begin || kv.second.kv_end < srcs[i]->end)
        return fail(HS_ESTATE, "a source sequence lacks cache for its layers");
    }
  }
  const bool dst_has = !dst->seqs.empty();
  if (dst->begin != dst->end && !ref.empty() && !dst_has)
    return fail(HS_ESTATE, "target serves layers but holds none of the sequences");
  if (dst_has) {
    if (dst->seqs.size() != ref.size()) return fail(HS_ESTATE, "target holds different sequences");
    for (const auto& kv : dst->seqs) {
      auto it = ref.find(kv.first);
      if (it == ref.end() || it->second.n_tokens != kv.second.n_tokens)
        return fail(HS_ESTATE, "target holds different sequences");
    }
  }
  int64_t need_blocks = 0;
  if (!dst_has) {
    if ((int64_t)ref.size() > dst->opts.max_seqs) return fail(HS_ENOMEM, "no free sequence slots");
    for (const auto& kv : ref) {
      if (kv.second.n_tokens > dst->opts.max_ctx) return fail(HS_ESTATE, "sequence longer than target max_ctx");
      need_blocks += blocks_for(kv.second.n_tokens);
    }
    if (need_blocks > (int64_t)dst->free_blocks.size())
      return fail(HS_ENOMEM, "not enough free KV blocks in the target");
  }
  // the target's weights for the whole union must have been submitted
  const int save_b = dst->begin, save_e = dst->end;
  dst->begin = ub;
  dst->end = ue;
  std::vector<Need> ne, nl, nh;
  DeviceGuard dg(dst->device);
  hs_status r = gather_needs(dst, &ne, &nl, &nh);
  dst->begin = save_b;
  dst->end = save_e;
  if (r != HS_OK) return fail(HS_ESTATE, std::string("merge target: ") + hs_last_error());

  uint64_t n_units = 0;
  for (int i = 0; i < n_srcs; ++i)
    for (const auto& kv : srcs[i]->seqs)
      n_units += (uint64_t)(srcs[i]->end - srcs[i]->begin) * blocks_for(kv.second.n_tokens);
  r = desc_reserve(dst, n_units + 1);  // before any state changes
  if (r != HS_OK) return r;

  hipStream_t s = pick(dst, stream);
  r = begin_call(dst, s);
  if (r != HS_OK) return r;
  for (int i = 0; i < n_srcs; ++i) {
    r = begin_call(srcs[i], s);  // drain: order after all work of the source
    if (r != HS_OK) return r;
  }
  if (!dst_has) {
    for (const auto& kv : ref) {
      Seq q;
      q.n_tokens = kv.second.n_tokens;
      for (int b = 0; b < blocks_for(q.n_tokens); ++b) {
        q.blocks.push_back(dst->free_blocks.back());
        dst->free_blocks.pop_back();
      }
      q.kv_begin = q.kv_end = dst->begin == dst->end ? ub : dst->begin;
      dst->seqs.emplace(kv.first, std::move(q));
    }
  }
  Units u;
  for (int i = 0; i < n_srcs; ++i) {
    hs_stage* sr = srcs[i];
    for (int l = sr->begin; l < sr->end; ++l)
      for (const auto& kv : sr->seqs) {
        const Seq& qs = kv.second;
        const Seq& qd = dst->seqs.at(kv.first);
        for (int b = 0; b < blocks_for(qs.n_tokens); ++b) {
          u.src.push_back((uint64_t)(uintptr_t)pool(sr, l) + (uint64_t)qs.blocks[b] * sr->unit_bytes);
          u.dst.push_back((uint64_t)(uintptr_t)pool(dst, l) + (uint64_t)qd.blocks[b] * dst->unit_bytes);
          u.valid.push_back(kBlock);
        }
      }
  }
  r = copy_units(dst, u, 0, s);
  if (r != HS_OK) return r;
  for (auto& kv : dst->seqs) {
    kv.second.kv_begin = std::min(kv.second.kv_begin, ub);
    kv.second.kv_end = std::max(kv.second.kv_end, ue);
  }
  dst->begin = ub;
  dst->end = ue;
  r = end_call(dst, s);
  if (r != HS_OK) return r;
  for (int i = 0; i < n_srcs; ++i) {
    hs_stage* sr = srcs[i];
    std::vector<int64_t> ids;
    for (const auto& kv : sr->seqs) ids.push_back(kv.first);
    for (int64_t id : ids) (void)hs_seq_free(sr, id);
    r = end_call(sr, s);
    if (r != HS_OK) return r;
  }
  return HS_OK;
  ABI_END
}

// --------------------------------------------------------- pinned memory

extern "C" hs_status hs_host_alloc(uint64_t bytes, void** out) {
  ABI_BEGIN
  if (!out) return fail(HS_EINVAL, "null output");
  *out = nullptr;
  if (bytes == 0) return fail(HS_EINVAL, "zero-byte allocation");
  if (hipHostMalloc(out, bytes, hipHostMallocDefault) != hipSuccess || !*out) {
    (void)hipGetLastError();
    *out = nullptr;
    return fail(HS_ENOMEM, "hipHostMalloc of " + std::to_string(bytes) + " bytes failed");
  }
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_host_free(void* p) {
  ABI_BEGIN
  if (p && hipHostFree(p) != hipSuccess) return fail(HS_EHIP, "hipHostFree failed");
  return HS_OK;
  ABI_END
}

// ------------------------------------------------------------------ timing

extern "C" hs_status hs_stage_set_timing(hs_stage* st, int32_t enable) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  st->timing = enable != 0;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_set_timing_sites(hs_stage* st, const char* sites) {
  ABI_BEGIN
  if (!st) return fail(HS_EINVAL, "null stage");
  std::string list;
  if (sites && *sites) {
    for (const char* c = sites; *c; ++c)
      if (*c != ' ') list.push_back(*c);
    list = "," + list + ",";
  }
  st->timing_sites = list;
  return HS_OK;
  ABI_END
}

extern "C" hs_status hs_stage_read_timing(hs_stage* st, hs_kernel_stat* out, int32_t cap,
                                          int32_t* n) {
  ABI_BEGIN
  if (!st || !n || cap < 0 || (cap > 0 && !out)) return fail(HS_EINVAL, "bad arguments");
  hs_status r = hs_stage_sync(st);
  if (r != HS_OK) return r;
  DeviceGuard dg(st->device);
  for (auto& p : st->pending) {
    float ms = 0;
    HIPTRY(hipEventElapsedTime(&ms, p.a, p.b));
    Stat& s = st->stats[p.name + "@" + p.site];
    s.name = p.name;
    s.site = p.site;
    s.launches += 1;
    s.ms += ms;
    s.flops += p.flops;
    s.bytes += p.bytes;
    st->ev_pool.push_back(p.a);
    st->ev_pool.push_back(p.b);
  }
  st->pending.clear();
  int32_t i = 0;
  for (const auto& kv : st->stats) {
    if (i < cap) {
      hs_kernel_stat& o = out[i];
      memset(&o, 0, sizeof o);
      strncpy(o.name, kv.second.name.c_str(), sizeof(o.name) - 1);
      strncpy(o.site, kv.second.site.c_str(), sizeof(o.site) - 1);
      o.launches = kv.second.launches;
      o.total_ms = kv.second.ms;
      o.flops = kv.second.flops;
      o.bytes = kv.second.bytes;
    }
    ++i;
  }
  *n = i;
  st->stats.clear();
  return HS_OK;
  ABI_END
}
