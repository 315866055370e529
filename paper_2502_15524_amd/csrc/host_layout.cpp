// Weight-image layout, image packing, KV-blob header codec and the
// thread-local error message. Pure C++: no HIP calls.
#include <string.h>

#include <set>
#include <string>

#include "hs_host.h"

namespace hs {

static thread_local std::string g_err;

hs_status fail(hs_status code, const std::string& msg) {
  g_err = msg;
  return code;
}
void clear_error() { g_err.clear(); }

bool cfg_valid(const hs_model_cfg* c, std::string* why) {
  auto no = [&](const char* m) {
    if (why) *why = m;
    return false;
  };
  if (!c) return no("null model cfg");
  if (c->n_layers <= 0 || c->n_layers > 1024) return no("n_layers must be in 1..1024");
  if (c->hidden <= 0 || c->hidden % 64) return no("hidden must be a positive multiple of 64");
  if (c->hidden > 8192) return no("hidden above 8192 is not supported");
  if (c->head_dim != 64 && c->head_dim != 128) return no("head_dim must be 64 or 128");
  if (c->n_heads <= 0 || c->n_kv_heads <= 0 || c->n_heads % c->n_kv_heads)
    return no("n_heads must be a positive multiple of n_kv_heads");
  const int g = c->n_heads / c->n_kv_heads;
  if (g != 1 && g != 2 && g != 4) return no("n_heads / n_kv_heads must be 1, 2 or 4");
  if (c->ffn <= 0 || c->ffn % 16 || c->ffn > (1 << 17))
    return no("ffn must be a positive multiple of 16, at most 131072");
  if (c->vocab <= 0 || c->vocab % 16 || c->vocab > (1 << 20))
    return no("vocab must be a positive multiple of 16, at most 1048576");
  if (!(c->rms_eps > 0.f)) return no("rms_eps must be positive");
  if (!(c->rope_base > 1.f)) return no("rope_base must be above 1");
  return true;
}

hs_status build_layout(const hs_model_cfg& c, int32_t rb, int32_t re, ImageLayout* L) {
  std::string why;
  if (!cfg_valid(&c, &why)) return fail(HS_EINVAL, why);
  if (rb < 0 || re > c.n_layers || rb >= re)
    return fail(HS_EINVAL, "resident range must satisfy 0 <= begin < end <= n_layers");
  const uint64_t H = c.hidden, F = c.ffn, V = c.vocab;
  const uint64_t QKV = (uint64_t)(c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  const uint64_t QD = (uint64_t)c.n_heads * c.head_dim;
  *L = ImageLayout();
  L->rb = rb;
  L->re = re;
  uint64_t off = 0;
  auto put = [&](int32_t layer, int32_t kind, uint64_t rows, uint64_t cols) {
    off = align_up(off, kAlign);
    const bool tiled = !(kind == HS_W_EMBED || kind == HS_W_ATTN_NORM ||
                         kind == HS_W_FFN_NORM || kind == HS_W_FINAL_NORM);
    hs_tensor_desc d;
    d.offset = off;
    d.bytes = tiled ? tiled_bytes(rows, cols) : rows * cols * 2;
    d.layer = layer;
    d.kind = kind;
    d.rows = (int64_t)rows;
    d.cols = (int64_t)cols;
    d.tiled = tiled ? 1 : 0;
    d.reserved = 0;
    L->descs.push_back(d);
    off += d.bytes;
    return d.offset;
  };
  if (rb == 0) {
    L->has_embed = true;
    L->embed = put(-1, HS_W_EMBED, V, H);
    L->embed_end = off;
  }
  for (int32_t l = rb; l < re; ++l) {
    LayerSlots s;
    s.attn_norm = put(l, HS_W_ATTN_NORM, 1, H);
    s.begin = s.attn_norm;
    s.qkv = put(l, HS_W_QKV, QKV, H);
    s.o = put(l, HS_W_O, H, QD);
    s.ffn_norm = put(l, HS_W_FFN_NORM, 1, H);
    s.gateup = put(l, HS_W_GATEUP, 2 * F, H);
    s.down = put(l, HS_W_DOWN, H, F);
    s.end = off;
    L->layers.push_back(s);
  }
  if (re == c.n_layers) {
    L->has_head = true;
    L->final_norm = put(-1, HS_W_FINAL_NORM, 1, H);
    L->head_begin = L->final_norm;
    L->lm_head = put(-1, HS_W_LM_HEAD, V, H);
    L->head_end = off;
  }
  L->bytes = align_up(off, kAlign);
  return HS_OK;
}

// --------------------------------------------------------------- KV blob

uint64_t blob_unit_bytes(int32_t n_kv, int32_t head_dim, int32_t block_size) {
  return 2ull * (uint64_t)n_kv * (uint64_t)block_size * (uint64_t)head_dim * 2ull;
}

void blob_sizes(BlobHeader* h, const std::vector<BlobRecord>& recs) {
  uint64_t blocks = 0;
  for (const auto& r : recs) blocks += (uint64_t)r.n_blocks;
  h->n_seqs = (int32_t)recs.size();
  h->payload_offset = align_up(kBlobHeader + kBlobRecord * recs.size(), 256);
  h->payload_bytes = (uint64_t)(h->layer_end - h->layer_begin) * blocks *
                     blob_unit_bytes(h->n_kv_heads, h->head_dim, h->block_size);
  h->total_bytes = h->payload_offset + h->payload_bytes;
}

template <typename T>
static void wr(uint8_t* p, uint64_t off, T v) {
  memcpy(p + off, &v, sizeof(T));
}
template <typename T>
static T rd(const uint8_t* p, uint64_t off) {
  T v;
  memcpy(&v, p + off, sizeof(T));
  return v;
}

std::vector<uint8_t> blob_encode_head(const BlobHeader& h, const std::vector<BlobRecord>& recs) {
  std::vector<uint8_t> b(h.payload_offset, 0);
  memcpy(b.data(), "HSKV", 4);
  wr<uint32_t>(b.data(), 4, kBlobVersion);
  wr<uint32_t>(b.data(), 8, kBlobDtypeBf16);
  wr<int32_t>(b.data(), 12, h.layer_begin);
  wr<int32_t>(b.data(), 16, h.layer_end);
  wr<int32_t>(b.data(), 20, h.n_kv_heads);
  wr<int32_t>(b.data(), 24, h.head_dim);
  wr<int32_t>(b.data(), 28, h.block_size);
  wr<int32_t>(b.data(), 32, (int32_t)recs.size());
  wr<uint32_t>(b.data(), 36, 0);
  wr<uint64_t>(b.data(), 40, h.payload_offset);
  wr<uint64_t>(b.data(), 48, h.payload_bytes);
  wr<uint64_t>(b.data(), 56, h.total_bytes);
  for (size_t i = 0; i < recs.size(); ++i) {
    const uint64_t o = kBlobHeader + kBlobRecord * i;
    wr<int64_t>(b.data(), o, recs[i].seq_id);
    wr<int32_t>(b.data(), o + 8, recs[i].n_tokens);
    wr<int32_t>(b.data(), o + 12, recs[i].n_blocks);
  }
  return b;
}

hs_status blob_decode_head(const void* pv, uint64_t avail, BlobHeader* h,
                           std::vector<BlobRecord>* recs) {
  const uint8_t* p = static_cast<const uint8_t*>(pv);
  if (!p) return fail(HS_EINVAL, "null blob");
  if (avail < kBlobHeader) return fail(HS_EINVAL, "blob shorter than its 64-byte header");
  if (memcmp(p, "HSKV", 4) != 0) return fail(HS_EINVAL, "bad blob magic");
  if (rd<uint32_t>(p, 4) != kBlobVersion) return fail(HS_EINVAL, "unsupported blob version");
  if (rd<uint32_t>(p, 8) != kBlobDtypeBf16) return fail(HS_EINVAL, "unsupported blob dtype");
  BlobHeader x;
  x.layer_begin = rd<int32_t>(p, 12);
  x.layer_end = rd<int32_t>(p, 16);
  x.n_kv_heads = rd<int32_t>(p, 20);
  x.head_dim = rd<int32_t>(p, 24);
  x.block_size = rd<int32_t>(p, 28);
  x.n_seqs = rd<int32_t>(p, 32);
  x.payload_offset = rd<uint64_t>(p, 40);
  x.payload_bytes = rd<uint64_t>(p, 48);
  x.total_bytes = rd<uint64_t>(p, 56);
  if (x.layer_begin < 0 || x.layer_end <= x.layer_begin || x.layer_end > (1 << 20))
    return fail(HS_EINVAL, "bad blob layer range");
  if (x.n_kv_heads <= 0 || x.n_kv_heads > 4096 || x.head_dim <= 0 || x.head_dim > 4096 ||
      x.block_size <= 0 || x.block_size > 4096)
    return fail(HS_EINVAL, "bad blob geometry");
  if (x.n_seqs < 0 || x.n_seqs > (1 << 24)) return fail(HS_EINVAL, "bad blob sequence count");
  if (avail < kBlobHeader + kBlobRecord * (uint64_t)x.n_seqs)
    return fail(HS_EINVAL, "blob truncated inside its sequence records");
  std::vector<BlobRecord> r((size_t)x.n_seqs);
  std::set<int64_t> ids;
  for (int32_t i = 0; i < x.n_seqs; ++i) {
    const uint64_t o = kBlobHeader + kBlobRecord * (uint64_t)i;
    r[i].seq_id = rd<int64_t>(p, o);
    r[i].n_tokens = rd<int32_t>(p, o + 8);
    r[i].n_blocks = rd<int32_t>(p, o + 12);
    if (r[i].n_tokens <= 0) return fail(HS_EINVAL, "blob record with no tokens");
    if ((int64_t)r[i].n_blocks != ((int64_t)r[i].n_tokens + x.block_size - 1) / x.block_size)
      return fail(HS_EINVAL, "blob record block count does not match its token count");
    if (!ids.insert(r[i].seq_id).second) return fail(HS_EINVAL, "blob repeats a sequence id");
  }
  // the payload must be representable: layers x blocks x unit bytes below
  // 2^62 (computed without wrapping), before blob_sizes forms it in 64 bits
  {
    unsigned __int128 blocks = 0;
    for (const BlobRecord& rc : r) blocks += (uint64_t)rc.n_blocks;
    const unsigned __int128 pay = (unsigned __int128)(uint64_t)(x.layer_end - x.layer_begin) *
                                  blocks *
                                  blob_unit_bytes(x.n_kv_heads, x.head_dim, x.block_size);
    if (pay >> 62) return fail(HS_EINVAL, "blob payload size out of range");
  }
  BlobHeader want = x;
  blob_sizes(&want, r);
  if (want.payload_offset != x.payload_offset || want.payload_bytes != x.payload_bytes ||
      want.total_bytes != x.total_bytes)
    return fail(HS_EINVAL, "blob size fields are inconsistent");
  if (h) *h = x;
  if (recs) *recs = std::move(r);
  return HS_OK;
}

}  // namespace hs

// ------------------------------------------------------------- C ABI (host)

using namespace hs;

extern "C" hs_status hs_weight_layout(const hs_model_cfg* cfg, int32_t rb, int32_t re,
                                      hs_tensor_desc* out, int32_t cap, int32_t* n,
                                      uint64_t* image_bytes) {
  try {
    if (!cfg) return fail(HS_EINVAL, "null model cfg");
    if (cap < 0 || (cap > 0 && !out)) return fail(HS_EINVAL, "bad output capacity");
    ImageLayout L;
    hs_status st = build_layout(*cfg, rb, re, &L);
    if (st != HS_OK) return st;
    const int32_t total = (int32_t)L.descs.size();
    for (int32_t i = 0; i < total && i < cap; ++i) out[i] = L.descs[i];
    if (n) *n = total;
    if (image_bytes) *image_bytes = L.bytes;
    return HS_OK;
  } catch (...) {
    return fail(HS_ENOMEM, "host allocation failed");
  }
}

namespace {
// Stored row of row i of a q or k projection with heads of d rows: inside a
// head, row 16 j + r of the first half goes to 32 j + r and its RoPE partner
// (the same row of the second half) to 32 j + 16 + r.
uint64_t qk_row(uint64_t i, uint64_t d) {
  const uint64_t h = i / d, r = i % d, half = d / 2;
  return h * d + ((r % half) / 16) * 32 + (r / half) * 16 + r % 16;
}
}  // namespace

extern "C" hs_status hs_image_put(const hs_model_cfg* cfg, int32_t rb, int32_t re, int32_t layer,
                                  int32_t src_kind, const uint16_t* src, uint64_t n_elems,
                                  void* image) {
  try {
    if (!cfg || !src || !image) return fail(HS_EINVAL, "null argument");
    ImageLayout L;
    hs_status st = build_layout(*cfg, rb, re, &L);
    if (st != HS_OK) return st;
    const uint64_t H = cfg->hidden, F = cfg->ffn, V = cfg->vocab, D = cfg->head_dim;
    const uint64_t QD = (uint64_t)cfg->n_heads * D, KD = (uint64_t)cfg->n_kv_heads * D;
    uint8_t* img = static_cast<uint8_t*>(image);
    const bool per_layer = !(src_kind == HS_SRC_EMBED || src_kind == HS_SRC_FINAL_NORM ||
                             src_kind == HS_SRC_LM_HEAD);
    const LayerSlots* ls = nullptr;
    if (per_layer) {
      if (layer < rb || layer >= re) return fail(HS_EINVAL, "layer is not resident in this image");
      ls = &L.layers[layer - rb];
    }
    auto copy_rows = [&](uint64_t dst_off, uint64_t rows, uint64_t cols) -> hs_status {
      if (n_elems != rows * cols) return fail(HS_EINVAL, "element count does not match the tensor shape");
      memcpy(img + dst_off, src, rows * cols * 2);
      return HS_OK;
    };
    // n_rows source rows into a tiled matrix of `rows` rows, row i -> map(i)
    auto tile = [&](uint64_t dst_off, uint64_t rows, uint64_t n_rows, uint64_t cols,
                    auto map) -> hs_status {
      if (n_elems != n_rows * cols) return fail(HS_EINVAL, "element count does not match the tensor shape");
      tile_rows(src, n_rows, cols, rows, img + dst_off, map);
      return HS_OK;
    };
    const uint64_t NQKV = QD + 2 * KD;
    switch (src_kind) {
      case HS_SRC_EMBED:
        if (!L.has_embed) return fail(HS_EINVAL, "image has no embedding");
        return copy_rows(L.embed, V, H);
      case HS_SRC_FINAL_NORM:
        if (!L.has_head) return fail(HS_EINVAL, "image has no final norm");
        return copy_rows(L.final_norm, 1, H);
      case HS_SRC_LM_HEAD:
        if (!L.has_head) return fail(HS_EINVAL, "image has no LM head");
        return tile(L.lm_head, V, V, H, [](uint64_t i) { return i; });
      case HS_SRC_ATTN_NORM: return copy_rows(ls->attn_norm, 1, H);
      case HS_SRC_FFN_NORM: return copy_rows(ls->ffn_norm, 1, H);
      // q and k heads: the two RoPE halves interleaved in groups of 16 rows
      case HS_SRC_WQ: return tile(ls->qkv, NQKV, QD, H, [&](uint64_t i) { return qk_row(i, D); });
      case HS_SRC_WK:
        return tile(ls->qkv, NQKV, KD, H, [&](uint64_t i) { return QD + qk_row(i, D); });
      case HS_SRC_WV: return tile(ls->qkv, NQKV, KD, H, [&](uint64_t i) { return QD + KD + i; });
      case HS_SRC_WO: return tile(ls->o, H, H, QD, [](uint64_t i) { return i; });
      case HS_SRC_WDOWN: return tile(ls->down, H, H, F, [](uint64_t i) { return i; });
      case HS_SRC_WGATE:
        return tile(ls->gateup, 2 * F, F, H, [](uint64_t f) { return (f / 16) * 32 + f % 16; });
      case HS_SRC_WUP:
        return tile(ls->gateup, 2 * F, F, H, [](uint64_t f) { return (f / 16) * 32 + 16 + f % 16; });
      default: return fail(HS_EINVAL, "unknown source tensor kind");
    }
  } catch (...) {
    return fail(HS_ENOMEM, "host allocation failed");
  }
}

extern "C" hs_status hs_pack_tiled(const uint16_t* src, int64_t rows, int64_t cols, void* dst) {
  if (!src || !dst) return fail(HS_EINVAL, "null argument");
  if (rows <= 0 || cols <= 0 || rows % 8) return fail(HS_EINVAL, "rows must be a positive multiple of 8");
  tile_rows(src, (uint64_t)rows, (uint64_t)cols, (uint64_t)rows, static_cast<uint8_t*>(dst),
            [](uint64_t i) { return i; });
  return HS_OK;
}

extern "C" hs_status hs_kv_blob_describe(const void* host_blob, uint64_t avail,
                                         hs_kv_blob_info* out) {
  try {
    BlobHeader h;
    hs_status st = blob_decode_head(host_blob, avail, &h, nullptr);
    if (st != HS_OK) return st;
    if (out) {
      out->layer_begin = h.layer_begin;
      out->layer_end = h.layer_end;
      out->n_kv_heads = h.n_kv_heads;
      out->head_dim = h.head_dim;
      out->block_size = h.block_size;
      out->n_seqs = h.n_seqs;
      out->payload_offset = h.payload_offset;
      out->payload_bytes = h.payload_bytes;
      out->total_bytes = h.total_bytes;
    }
    return HS_OK;
  } catch (...) {
    return fail(HS_ENOMEM, "host allocation failed");
  }
}

extern "C" const char* hs_last_error(void) { return hs::g_err.c_str(); }
