// Host-only internals of the engine: weight-image layout, KV-blob codec and
// error reporting. No HIP here, so these parts build and run without a GPU.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/hs.h"

namespace hs {

// Thread-local error message + status helper.
hs_status fail(hs_status code, const std::string& msg);
void clear_error();

bool cfg_valid(const hs_model_cfg* c, std::string* why);

constexpr uint64_t kAlign = 256;
inline uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Byte ranges of one resident layer's tensors inside the image.
struct LayerSlots {
  uint64_t begin, end;  // whole layer
  uint64_t attn_norm, qkv, o, ffn_norm, gateup, down;
};

struct ImageLayout {
  int32_t rb = 0, re = 0;
  bool has_embed = false, has_head = false;
  uint64_t embed = 0, embed_end = 0;       // embedding range
  uint64_t head_begin = 0, head_end = 0;   // final norm + LM head range
  uint64_t final_norm = 0, lm_head = 0;
  std::vector<LayerSlots> layers;          // index = layer - rb
  std::vector<hs_tensor_desc> descs;
  uint64_t bytes = 0;
};

// Fails with HS_EINVAL on an invalid cfg or range.
hs_status build_layout(const hs_model_cfg& cfg, int32_t rb, int32_t re, ImageLayout* out);

// Tiled matrix format (see hs.h): byte offset of element (row, col) of a
// matrix with `rows` rows, and its total size for `cols` columns.
inline uint64_t round64(uint64_t x) { return (x + 63) / 64 * 64; }
inline uint64_t tiled_bytes(uint64_t rows, uint64_t cols) { return rows * round64(cols) * 2; }
inline uint64_t tiled_offset(uint64_t rows, uint64_t row, uint64_t col) {
  const uint64_t kb = col / 64, nb = row / 8, r = row % 8, c = (col % 64) / 8;
  return (kb * (rows / 8) + nb) * 1024 + r * 128 + ((c ^ r) * 16) + (col % 8) * 2;
}
// Copy row-major rows [0, n_rows) of src ([n_rows][cols]) into the tiled
// matrix `dst` (total `rows` rows) at destination rows dst_row(i).
template <typename RowMap>
void tile_rows(const uint16_t* src, uint64_t n_rows, uint64_t cols, uint64_t rows, uint8_t* dst,
               RowMap dst_row) {
  for (uint64_t i = 0; i < n_rows; ++i) {
    const uint64_t r = dst_row(i);
    for (uint64_t c = 0; c < round64(cols); c += 8) {  // columns past cols are zero
      const uint64_t n = c >= cols ? 0 : (cols - c < 8 ? cols - c : 8);
      uint8_t* d = dst + tiled_offset(rows, r, c);
      if (n) __builtin_memcpy(d, src + i * cols + c, n * 2);
      if (n < 8) __builtin_memset(d + n * 2, 0, (8 - n) * 2);
    }
  }
}

// --------------------------------------------------------------- KV blob

constexpr uint32_t kBlobVersion = 1;
constexpr uint32_t kBlobDtypeBf16 = 1;
constexpr uint64_t kBlobHeader = 64;
constexpr uint64_t kBlobRecord = 16;

struct BlobRecord {
  int64_t seq_id;
  int32_t n_tokens;
  int32_t n_blocks;
};

struct BlobHeader {
  int32_t layer_begin, layer_end, n_kv_heads, head_dim, block_size, n_seqs;
  uint64_t payload_offset, payload_bytes, total_bytes;
};

uint64_t blob_unit_bytes(int32_t n_kv, int32_t head_dim, int32_t block_size);
// Fills payload_offset / payload_bytes / total_bytes from the other fields.
void blob_sizes(BlobHeader* h, const std::vector<BlobRecord>& recs);
// Header + records + zero padding up to payload_offset.
std::vector<uint8_t> blob_encode_head(const BlobHeader& h, const std::vector<BlobRecord>& recs);
// Parses and validates the start of a blob (`avail` bytes available).
hs_status blob_decode_head(const void* p, uint64_t avail, BlobHeader* h,
                           std::vector<BlobRecord>* recs);

}  // namespace hs
