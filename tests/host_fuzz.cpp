// Randomised checks of the engine's host-only code (weight-image layout,
// tiled packing, KV-blob header codec), built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitize.py. Stops at the
// first failure: a sanitizer report aborts the process, and every property
// violation prints what failed and exits non-zero.
//
// Properties:
//  * blob headers: a header encoded from valid fields decodes to the same
//    fields; after random byte flips, field overwrites with extreme values
//    and truncations, the decoder either rejects the bytes or returns fields
//    whose sizes are exactly consistent (computed here in 128-bit
//    arithmetic) and lie inside the bytes it was given;
//  * layouts: for random model shapes and layer ranges, every tensor lies
//    inside the image, tensors do not overlap, each decoder layer is one
//    contiguous byte range holding its tensors;
//  * tiled packing writes exactly rows * round64(cols) * 2 bytes.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "../paper_2502_15524_amd/csrc/hs_host.h"

using namespace hs;

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next() {  // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
int64_t pick(int64_t lo, int64_t hi) { return lo + (int64_t)(next() % (uint64_t)(hi - lo + 1)); }

[[noreturn]] void die(const char* what, uint64_t iter) {
  fprintf(stderr, "FAIL at case %llu: %s\n", (unsigned long long)iter, what);
  exit(1);
}

typedef unsigned __int128 u128;

// Field values a mutation may write: boundaries and random bits.
int64_t extreme() {
  static const int64_t v[] = {0, 1, -1, 2, 15, 16, 17, 255, 256, 4096, 4097, 65536,
                              INT32_MAX, INT32_MIN, (int64_t)INT32_MAX + 1, INT64_MAX, INT64_MIN,
                              (int64_t)1 << 40, 1 << 20, (1 << 20) + 1, 1 << 24, (1 << 24) + 1};
  if (next() % 4 == 0) return (int64_t)next();
  return v[next() % (sizeof v / sizeof v[0])];
}

void check_blob(uint64_t iter) {
  BlobHeader h{};
  h.layer_begin = (int32_t)pick(0, 40);
  h.layer_end = h.layer_begin + (int32_t)pick(1, 8);
  h.n_kv_heads = (int32_t)pick(1, 64);
  h.head_dim = next() % 2 ? 64 : 128;
  h.block_size = 16;
  std::vector<BlobRecord> recs((size_t)pick(0, 40));
  for (size_t i = 0; i < recs.size(); ++i) {
    recs[i].seq_id = (int64_t)(next() >> 1) ^ (int64_t)i;
    recs[i].n_tokens = (int32_t)pick(1, 5000);
    recs[i].n_blocks = (recs[i].n_tokens + 15) / 16;
  }
  std::sort(recs.begin(), recs.end(),
            [](const BlobRecord& a, const BlobRecord& b) { return a.seq_id < b.seq_id; });
  recs.erase(std::unique(recs.begin(), recs.end(),
                         [](const BlobRecord& a, const BlobRecord& b) {
                           return a.seq_id == b.seq_id;
                         }),
             recs.end());
  blob_sizes(&h, recs);
  std::vector<uint8_t> b = blob_encode_head(h, recs);
  // the untouched header round-trips
  {
    BlobHeader g;
    std::vector<BlobRecord> r;
    if (blob_decode_head(b.data(), b.size(), &g, &r) != HS_OK) die("valid header rejected", iter);
    if (g.layer_begin != h.layer_begin || g.layer_end != h.layer_end ||
        g.n_kv_heads != h.n_kv_heads || g.head_dim != h.head_dim ||
        g.total_bytes != h.total_bytes || r.size() != recs.size())
      die("header fields changed in the round trip", iter);
  }
  // mutations
  const int kind = (int)(next() % 4);
  if (kind == 0) {  // byte flips
    for (int k = (int)pick(1, 8); k > 0; --k) b[next() % b.size()] ^= (uint8_t)(1 + next() % 255);
  } else if (kind == 1) {  // a header field overwritten
    const int off = (int)(4 * pick(1, 15));
    const int64_t v = extreme();
    memcpy(b.data() + off, &v, off >= 40 ? 8 : 4);
  } else if (kind == 2 && !recs.empty()) {  // a record field overwritten
    const uint64_t o = kBlobHeader + kBlobRecord * (next() % recs.size()) + 4 * pick(0, 3);
    const int64_t v = extreme();
    memcpy(b.data() + o, &v, 4);
  }
  // the bytes available: all, or a truncation
  uint64_t avail = b.size();
  if (next() % 3 == 0) avail = next() % (b.size() + 1);
  std::vector<uint8_t> buf(b.begin(), b.begin() + (long)avail);  // exact-size heap copy
  BlobHeader g;
  std::vector<BlobRecord> r;
  if (blob_decode_head(buf.data(), avail, &g, &r) != HS_OK) return;
  // accepted: everything must be consistent and inside the given bytes
  if (g.n_seqs < 0 || (uint64_t)g.n_seqs != r.size()) die("record count", iter);
  if (kBlobHeader + kBlobRecord * (u128)g.n_seqs > avail) die("records past the bytes", iter);
  if (g.layer_end <= g.layer_begin || g.layer_begin < 0) die("layer range", iter);
  if (g.block_size <= 0 || g.n_kv_heads <= 0 || g.head_dim <= 0) die("geometry", iter);
  u128 blocks = 0;
  for (const BlobRecord& x : r) {
    if (x.n_tokens <= 0) die("empty record accepted", iter);
    const u128 need = ((u128)x.n_tokens + (u128)g.block_size - 1) / (u128)g.block_size;
    if ((u128)(uint32_t)x.n_blocks != need || x.n_blocks < 0) die("block count", iter);
    blocks += (u128)x.n_blocks;
  }
  const u128 unit = (u128)2 * (u128)g.n_kv_heads * (u128)g.block_size * (u128)g.head_dim * 2;
  const u128 payload = (u128)(g.layer_end - g.layer_begin) * blocks * unit;
  const u128 off = ((kBlobHeader + kBlobRecord * (u128)g.n_seqs) + 255) / 256 * 256;
  if ((u128)g.payload_offset != off) die("payload offset", iter);
  if ((u128)g.payload_bytes != payload) die("payload size wrapped or wrong", iter);
  if ((u128)g.total_bytes != off + payload) die("total size wrapped or wrong", iter);
  hs_kv_blob_info info;
  if (hs_kv_blob_describe(buf.data(), avail, &info) != HS_OK) die("describe disagrees", iter);
  if (info.total_bytes != g.total_bytes) die("describe total", iter);
}

void check_layout(uint64_t iter) {
  hs_model_cfg c{};
  c.n_layers = (int32_t)pick(0, 48);
  c.head_dim = next() % 2 ? 64 : 128;
  const int g = 1 << pick(0, 2);
  c.n_kv_heads = (int32_t)pick(0, 16);
  c.n_heads = c.n_kv_heads * g;
  c.hidden = (int32_t)(64 * pick(0, 80));
  c.ffn = (int32_t)(16 * pick(0, 900));
  c.vocab = (int32_t)(16 * pick(0, 9000));
  c.rms_eps = 1e-5f;
  c.rope_base = 10000.f;
  if (next() % 8 == 0) {  // an invalid field
    const int64_t v = extreme();
    switch (next() % 5) {
      case 0: c.hidden = (int32_t)v; break;
      case 1: c.n_heads = (int32_t)v; break;
      case 2: c.ffn = (int32_t)v; break;
      case 3: c.vocab = (int32_t)v; break;
      default: c.n_layers = (int32_t)v; break;
    }
  }
  const int64_t nl = std::min<int64_t>(c.n_layers, 2000);
  const int32_t rb = (int32_t)pick(-2, nl + 1), re = (int32_t)pick(-2, nl + 2);
  int32_t n = 0;
  uint64_t bytes = 0;
  if (hs_weight_layout(&c, rb, re, nullptr, 0, &n, &bytes) != HS_OK) return;
  std::vector<hs_tensor_desc> d((size_t)n);
  int32_t n2 = 0;
  if (hs_weight_layout(&c, rb, re, d.data(), n, &n2, &bytes) != HS_OK || n2 != n)
    die("layout changed between calls", iter);
  std::sort(d.begin(), d.end(),
            [](const hs_tensor_desc& a, const hs_tensor_desc& b) { return a.offset < b.offset; });
  uint64_t end = 0;
  for (const hs_tensor_desc& t : d) {
    if (t.bytes == 0) die("empty tensor", iter);
    if (t.offset < end) die("tensors overlap", iter);
    if (t.offset + t.bytes < t.offset || t.offset + t.bytes > bytes) die("tensor past the image", iter);
    end = t.offset + t.bytes;
  }
  // each decoder layer's tensors form one contiguous run (no other tensor
  // inside): in offset order, a layer index >= 0 never reappears after
  // another one (-1 marks the embedding at the start and the final norm and
  // head at the end)
  std::vector<int32_t> seen;
  for (size_t i = 0; i < d.size(); ++i)
    if (d[i].layer >= 0 && (i == 0 || d[i].layer != d[i - 1].layer)) {
      if (std::find(seen.begin(), seen.end(), d[i].layer) != seen.end())
        die("layer split into several byte ranges", iter);
      seen.push_back(d[i].layer);
    }
}

void check_pack(uint64_t iter) {
  const int64_t rows = 8 * pick(1, 6), cols = pick(1, 200);
  std::vector<uint16_t> src((size_t)(rows * cols));
  for (auto& v : src) v = (uint16_t)next();
  const size_t out = (size_t)rows * (size_t)((cols + 63) / 64 * 64) * 2;
  std::vector<uint8_t> dst(out);  // exact size: ASan flags any write past it
  if (hs_pack_tiled(src.data(), rows, cols, dst.data()) != HS_OK) die("pack rejected", iter);
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t k = 0; k < cols; ++k) {
      uint16_t v;
      memcpy(&v, dst.data() + tiled_offset((uint64_t)rows, (uint64_t)r, (uint64_t)k), 2);
      if (v != src[(size_t)(r * cols + k)]) die("packed element misplaced", iter);
    }
  if (hs_pack_tiled(src.data(), rows + 1, cols, dst.data()) == HS_OK) die("odd rows accepted", iter);
}

}  // namespace

int main(int argc, char** argv) {
  const uint64_t n = argc > 1 ? strtoull(argv[1], nullptr, 10) : 20000;
  for (uint64_t i = 0; i < n; ++i) {
    check_blob(i);
    if (i % 4 == 0) check_layout(i);
    if (i % 16 == 0) check_pack(i);
  }
  printf("ok %llu cases\n", (unsigned long long)n);
  return 0;
}
