/*
 * hs.h - C ABI of the pipeline-stage engine (one GPU, gfx950).
 *
 * A stage hosts a contiguous range of decoder layers of a Llama-style model
 * (paper, section 2.1 and section 4.1: pipeline parallelism gives each worker
 * a contiguous slice of layers and passes intermediate results between
 * workers in order). It receives its weights as a stream of byte chunks from
 * pinned host memory and uses them in place (section 5.2, parameter manager:
 * zero-copy, pipelined, several streams), runs prefill and KV-cached decode
 * (section 2.1), and exports / imports its paged KV cache so that stages can
 * be consolidated into one worker (section 6.1 scaling down, section 6.2 KV
 * cache migration).
 *
 * Conventions for every call:
 *  - Return value: HS_OK or a negative hs_status. hs_last_error() returns a
 *    thread-local message for the last failure on the calling thread.
 *  - Arguments and state are validated before anything is enqueued. A call
 *    that fails changes no state, except HS_EHIP, which reports a HIP
 *    runtime failure (possibly from earlier asynchronous work).
 *  - `stream` is a hipStream_t passed as void*; NULL is the null (default)
 *    stream. Calls on one stage are ordered with each other even when they
 *    use different streams (each call waits for the previous one).
 *    Work is asynchronous: results are valid once `stream` has reached the
 *    end of the call's work (hipStreamSynchronize, an event, or
 *    hs_stage_sync).
 *  - Device buffers passed in (in/out/logits/blobs) are owned by the caller
 *    and must stay valid until that work completes; the library keeps no
 *    caller pointer after returning, except `pinned_src` of
 *    hs_stage_load_chunk, which must stay valid until the chunk has landed.
 *  - A stage may be driven from one thread at a time; different stages may
 *    be driven from different threads.
 *  - Every stream the library creates has the default priority.
 */
#ifndef HS_H
#define HS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hs_stage hs_stage; /* opaque; owned by the library */

typedef enum {
  HS_OK = 0,
  HS_EINVAL = -1,    /* bad argument, shape, id or blob */
  HS_ENOMEM = -2,    /* device memory, KV blocks or sequence slots exhausted */
  HS_ENOTREADY = -3, /* weights of a needed layer were never submitted */
  HS_ERANGE = -4,    /* caller buffer too small (required size returned) */
  HS_ESTATE = -5,    /* call not valid in the stage's current state */
  HS_EHIP = -6       /* HIP runtime error */
} hs_status;

/* Model shape. Llama-style decoder: pre-norm RMSNorm (eps), rotate-half
 * RoPE (base), causal grouped-query attention with n_heads query heads over
 * n_kv_heads KV heads (query head h reads KV head h / (n_heads/n_kv_heads)),
 * SwiGLU FFN of width ffn, no biases, untied LM head. head_dim must be 64
 * or 128, n_heads / n_kv_heads 1, 2 or 4; hidden a multiple of 64 (at most
 * 8192), ffn and vocab multiples of 16 (at most 131072 and 1048576),
 * n_layers at most 1024. */
typedef struct {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
  float rms_eps, rope_base;
} hs_model_cfg;

/* Stage options. All sizes are upper bounds fixed at creation. */
typedef struct {
  /* Layers whose weights the stage holds: a superset of the serving range
   * (a "full-memory" worker holds more than it serves, section 4.1).
   * resident_end == 0 means "same as the serving range". */
  int32_t resident_begin, resident_end;
  int32_t max_seqs;         /* live sequences (>= 1) */
  int32_t max_ctx;          /* tokens per sequence, prompt + decode (>= 1) */
  int32_t max_batch_tokens; /* tokens in one prefill call (>= 1) */
  int32_t kv_block_size;    /* tokens per KV block; must be 16 */
  int32_t kv_num_blocks;    /* 0 = max_seqs * ceil(max_ctx / kv_block_size) */
  int32_t n_copy_streams;   /* weight-upload streams, 1..8 */
} hs_stage_opts;

/* ------------------------------------------------------------------------
 * Weight image (host-side, no GPU needed).
 *
 * The stage's weights are one packed byte image in a layout the library
 * defines (the counterpart of the prefetcher's shared-memory model file,
 * section 5.1). Every tensor is bf16 and 256-byte aligned, and the tensors of
 * one layer are contiguous, so a layer is usable as soon as one byte range
 * has landed. Order: embedding (if the resident range starts at layer 0),
 * then each resident layer, then the final norm and LM head (if it ends at
 * the last layer).
 *
 * Tiled matrices. The projection matrices (QKV, O, gate/up, down, LM head),
 * logically [rows][cols] with cols the input dimension, are stored as 1 KiB
 * blocks of 8 rows x 64 columns: with Kp = cols rounded up to 64, block
 * (kb, nb) covers rows 8 nb .. 8 nb + 7 and columns 64 kb .. 64 kb + 63 and
 * sits at byte offset (kb * rows / 8 + nb) * 1024 (column blocks outermost).
 * Inside a block, row r (0..7) fills bytes [128 r, 128 r + 128), and its
 * 16-byte chunk c (columns 64 kb + 8 c .. + 7) is stored at position c ^ r.
 * Columns cols .. Kp - 1 are zero. A 64-column slab of any row range is then
 * one contiguous run of bytes, in the order the GEMM kernels consume it.
 * Embedding and norm gains are plain row-major.
 */
typedef enum {
  HS_W_EMBED = 0,      /* [vocab][hidden] */
  HS_W_ATTN_NORM = 1,  /* [hidden] RMSNorm gain before attention */
  HS_W_QKV = 2,        /* [(n_heads + 2 n_kv_heads) head_dim][hidden]: q, k, v rows;
                          inside each q and k head the two RoPE halves are
                          interleaved in groups of 16 rows (rows 16j..16j+15 of
                          the first half, then the same rows of the second) */
  HS_W_O = 3,          /* [hidden][n_heads head_dim] */
  HS_W_FFN_NORM = 4,   /* [hidden] RMSNorm gain before the FFN */
  HS_W_GATEUP = 5,     /* [2 ffn][hidden]: gate and up rows interleaved in
                          groups of 16 (16 gate rows, then the same 16 up rows) */
  HS_W_DOWN = 6,       /* [hidden][ffn] */
  HS_W_FINAL_NORM = 7, /* [hidden] */
  HS_W_LM_HEAD = 8     /* [vocab][hidden] */
} hs_weight_kind;

typedef struct {
  uint64_t offset, bytes; /* byte range inside the image */
  int32_t layer;          /* decoder layer; -1 for embedding, final norm, head */
  int32_t kind;           /* hs_weight_kind */
  int64_t rows, cols;     /* logical shape */
  int32_t tiled;          /* 1: tiled matrix format (bytes = rows * Kp * 2) */
  int32_t reserved;
} hs_tensor_desc;

/* Describe the image of resident layers [resident_begin, resident_end).
 * Writes min(cap, total) descriptors to `out` (may be NULL when cap == 0),
 * the total count to *n and the image size to *image_bytes.
 * Errors: HS_EINVAL for an invalid model or range. */
hs_status hs_weight_layout(const hs_model_cfg* cfg, int32_t resident_begin,
                           int32_t resident_end, hs_tensor_desc* out,
                           int32_t cap, int32_t* n, uint64_t* image_bytes);

/* Standard source tensors accepted by hs_image_put, each bf16 row-major in
 * the usual [out_features][in_features] orientation. */
typedef enum {
  HS_SRC_EMBED = 0, HS_SRC_ATTN_NORM = 1, HS_SRC_WQ = 2, HS_SRC_WK = 3,
  HS_SRC_WV = 4, HS_SRC_WO = 5, HS_SRC_FFN_NORM = 6, HS_SRC_WGATE = 7,
  HS_SRC_WUP = 8, HS_SRC_WDOWN = 9, HS_SRC_FINAL_NORM = 10, HS_SRC_LM_HEAD = 11
} hs_src_kind;

/* Copy one standard tensor (bf16 bits, `n_elems` values) into a host image
 * laid out by hs_weight_layout for the same cfg and resident range.
 * `layer` is ignored for embedding, final norm and head. Host memory only;
 * the caller owns both buffers. Errors: HS_EINVAL if the tensor is not part
 * of this image or n_elems does not match its shape. */
hs_status hs_image_put(const hs_model_cfg* cfg, int32_t resident_begin,
                       int32_t resident_end, int32_t layer, int32_t src_kind,
                       const uint16_t* src, uint64_t n_elems, void* image);

/* Write a row-major bf16 matrix [rows][cols] (rows % 8 == 0) into the tiled
 * matrix format at dst (rows * Kp * 2 bytes, host memory, caller-owned).
 * Errors: HS_EINVAL for rows % 8 != 0 or a non-positive shape. */
hs_status hs_pack_tiled(const uint16_t* src, int64_t rows, int64_t cols, void* dst);

/* ------------------------------------------------------------------------
 * Stage lifecycle.
 */

/* Create a stage serving layers [layer_begin, layer_end) on HIP device
 * `device`. Allocates the device weight image (resident range), the paged
 * KV pools (one per resident layer, analytic size, section 7 startup
 * optimisations), activation workspace and streams. An empty serving range
 * (begin == end) is allowed when the resident range is not empty: such a
 * stage can only import KV or be the target of hs_stage_merge.
 * Errors: HS_EINVAL (cfg, ranges, opts), HS_ENOMEM, HS_EHIP. */
hs_status hs_stage_create(const hs_model_cfg* cfg, int32_t layer_begin,
                          int32_t layer_end, const hs_stage_opts* opts,
                          int32_t device, hs_stage** out);

/* Wait for all work of the stage, then free everything it owns. NULL is a
 * no-op. */
hs_status hs_stage_destroy(hs_stage* st);

/* Wait for all work the stage has enqueued (compute and weight upload).
 * Returns HS_EHIP if any of it failed. */
hs_status hs_stage_sync(hs_stage* st);

/* ------------------------------------------------------------------------
 * Streamed weight loading (section 5.1 and 5.2; overlap of loading with the
 * first inference is the refinement of the TTFT model of equation 5).
 */

/* Enqueue an asynchronous copy of `bytes` bytes from pinned host memory to
 * the device image at `image_offset` on one of the stage's copy streams
 * (round-robin), and record an event for it. Chunks must not overlap
 * chunks already submitted. Prefill and decode make each layer wait on the
 * events of the chunks that cover its bytes, so a layer computes as soon as
 * its weights land while later chunks are still in flight.
 * `pinned_src` must be page-locked (hipHostMalloc) and stay valid until the
 * chunk has landed (hs_stage_loaded or hs_stage_sync).
 * Overlap needs the copy streams on hardware queues of their own: HIP
 * spreads a process's streams over GPU_MAX_HW_QUEUES queues (4 by
 * default) and runs one queue's work in order, so a prefill whose stream
 * shares a queue with a copy stream starts only after every chunk queued
 * there. Set GPU_MAX_HW_QUEUES, before the HIP runtime starts, to at least
 * the number of streams in use (the stage's copy streams, the caller's
 * streams); 8 suffices for one loading stage and a few caller streams.
 * Errors: HS_EINVAL (range outside the image, overlap, NULL src), HS_EHIP. */
hs_status hs_stage_load_chunk(hs_stage* st, uint64_t image_offset,
                              const void* pinned_src, uint64_t bytes);

/* Non-blocking progress query: *layers_ready = number of leading resident
 * layers whose bytes have all landed; *watermark = length of the landed
 * prefix of the image (the device-side counterpart of the prefetcher's
 * "fetched up to" header, section 5.1). Either pointer may be NULL. */
hs_status hs_stage_loaded(hs_stage* st, int32_t* layers_ready,
                          uint64_t* watermark);

/* Forget every submitted chunk (after waiting for them), so the next
 * prefill needs the weights to be streamed again: a new cold start of the
 * same stage. KV content and sequences are kept. */
hs_status hs_stage_invalidate_weights(hs_stage* st);

/* ------------------------------------------------------------------------
 * Inference (section 2.1: prefill computes and caches the keys and values of
 * the prompt and produces the first token; decode reuses the cache and
 * produces one token per step).
 */

/* Prefill `n_seqs` new sequences. seq_ids (host, distinct, not live) name
 * them; seq_lens (host, each >= 1) give their prompt lengths; the total T
 * must not exceed max_batch_tokens, and each length max_ctx.
 *  in  : stage starts at layer 0 -> device int32 token ids [T];
 *        otherwise device bf16 hidden states [T][hidden], read in place
 *        by the stage's first layer (it may be `out` itself; otherwise the
 *        two must not overlap).
 *        Tokens and rows are packed sequence after sequence.
 *  out : stage ends at the last layer -> device int32 [n_seqs], the greedy
 *        next token of each sequence (lowest index among equal maxima);
 *        otherwise device bf16 [T][hidden], the residual stream after the
 *        stage's last layer (one 16-bit hidden vector per token, the
 *        inter-stage message of section 4.1).
 *  logits_opt : last stage only, optional device float32 [n_seqs][vocab],
 *        the logits of each sequence's last position.
 * Each layer waits on the upload events of its own weights only.
 * Errors: HS_EINVAL, HS_ENOMEM (blocks or sequence slots), HS_ENOTREADY
 * (a needed layer has bytes not covered by any submitted chunk), HS_ESTATE
 * (empty serving range), HS_EHIP. */
hs_status hs_stage_prefill(hs_stage* st, int32_t n_seqs, const int64_t* seq_ids,
                           const int32_t* seq_lens, const void* in, void* out,
                           float* logits_opt, void* stream);

/* One decode step for `n_seqs` live sequences (host seq_ids, distinct):
 * each gets one new position appended to its KV cache.
 *  in  : first stage -> device int32 [n_seqs] token ids; otherwise device
 *        bf16 [n_seqs][hidden] (as for prefill: read in place, `out` or
 *        not overlapping it).
 *  out : last stage -> device int32 [n_seqs] next tokens; otherwise device
 *        bf16 [n_seqs][hidden].
 *  logits_opt : as for prefill.
 * Errors: HS_EINVAL (unknown or repeated id), HS_ENOMEM (no free block),
 * HS_ERANGE (a sequence would exceed max_ctx), HS_ENOTREADY, HS_ESTATE
 * (empty serving range, or a sequence whose cache does not cover the
 * serving layers), HS_EHIP. */
hs_status hs_stage_decode(hs_stage* st, int32_t n_seqs, const int64_t* seq_ids,
                          const void* in, void* out, float* logits_opt,
                          void* stream);

/* Release a live sequence and its KV blocks. Errors: HS_EINVAL if unknown. */
hs_status hs_seq_free(hs_stage* st, int64_t seq_id);

/* Number of cached positions of a live sequence. HS_EINVAL if unknown. */
hs_status hs_seq_tokens(const hs_stage* st, int64_t seq_id, int32_t* n_tokens);

typedef struct {
  int32_t layer_begin, layer_end;       /* serving range */
  int32_t resident_begin, resident_end; /* weights held */
  int32_t live_seqs, free_blocks, total_blocks, block_size;
  uint64_t image_bytes, kv_bytes;       /* device bytes of weights and KV */
} hs_stage_info;

hs_status hs_stage_get_info(const hs_stage* st, hs_stage_info* out);

/* ------------------------------------------------------------------------
 * KV cache migration (section 6.2: stop scheduling, wait for in-flight
 * batches, take the blocks used by the live requests and gather them to
 * the worker that holds the whole model, placing them at the layers of the
 * worker they came from).
 *
 * Blob format (little-endian), the only serialized runtime state:
 *   0  "HSKV"   4 u32 version=1   8 u32 dtype=1 (bf16)
 *   12 i32 layer_begin  16 i32 layer_end  20 i32 n_kv_heads  24 i32 head_dim
 *   28 i32 block_size   32 i32 n_seqs     36 u32 0
 *   40 u64 payload_offset = align_up(64 + 16 n_seqs, 256)
 *   48 u64 payload_bytes  56 u64 total_bytes
 *   64 n_seqs records {i64 seq_id, i32 n_tokens, i32 n_blocks}, zero pad
 *   payload: per layer, per sequence (record order), per logical block:
 *            K block [n_kv][block_size][head_dim] then V block, bf16,
 *            post-RoPE keys; token slots past n_tokens are zero.
 */

/* Size of the blob hs_kv_export would write for these sequences over the
 * stage's serving layers. Errors: HS_EINVAL (unknown/repeated id),
 * HS_ESTATE (empty serving range). */
hs_status hs_kv_export_size(const hs_stage* st, int32_t n_seqs,
                            const int64_t* seq_ids, uint64_t* bytes);

/* Gather the KV blocks of the listed live sequences, for every layer the
 * stage serves, into `dst` (device memory, `cap` bytes). *written receives
 * the blob size; if cap is smaller, nothing is enqueued, *written holds the
 * required size and HS_ERANGE is returned. Bit-exact: a blob imported into
 * another stage and exported again is byte-identical.
 * Errors: HS_EINVAL (ids, dst not device memory), HS_ERANGE, HS_ESTATE,
 * HS_EHIP. */
hs_status hs_kv_export(hs_stage* st, int32_t n_seqs, const int64_t* seq_ids,
                       void* dst, uint64_t cap, uint64_t* written,
                       void* stream);

/* Scatter a blob (device memory, `bytes` long) into the stage's KV pools at
 * the blob's layers, which must be resident here. A sequence already live
 * in the stage must have the same token count and keeps its block table;
 * a new one gets fresh blocks. Reads the blob's header synchronously.
 * Errors: HS_EINVAL (malformed blob, geometry mismatch, layers not
 * resident, token-count mismatch), HS_ENOMEM (not enough free blocks or
 * sequence slots; nothing is written), HS_EHIP. */
hs_status hs_kv_import(hs_stage* st, const void* src, uint64_t bytes,
                       void* stream);

/* The first bytes of the blob hs_kv_export would write for these sequences
 * now (its 64-byte header, the per-sequence records and the zero padding up
 * to the payload), written to host memory `host_dst` (`cap` bytes; any host
 * memory). *written receives their length (payload_offset); HS_ERANGE if cap
 * is smaller. It lets a worker that exports hand the importer a host copy of
 * the blob's description with the device blob (section 6.2: the migration
 * thread sends the blocks' descriptions along with the blocks), so that the
 * import reads nothing back from the device. No GPU work.
 * Errors: HS_EINVAL (ids), HS_ERANGE. */
hs_status hs_kv_export_head(const hs_stage* st, int32_t n_seqs, const int64_t* seq_ids,
                            void* host_dst, uint64_t cap, uint64_t* written);

/* Import n_blobs device blobs in one call: one upload of copy descriptors
 * and one copy launch for all of them, no device-to-host read and no host
 * wait. srcs[i] (device memory, 16-byte aligned, bytes[i] long) is a blob
 * as hs_kv_export writes it; heads[i] (host memory, head_bytes[i] bytes) must
 * hold that blob's first bytes, at least its header and records, as
 * hs_kv_export_head returns them (the call trusts them to describe srcs[i]).
 * The blobs are applied in order: blob i is validated as hs_kv_import would
 * validate it after blobs 0 .. i-1, so blobs of adjacent layer ranges of the
 * same sequences (one per source stage) build up each sequence's cache.
 * Every blob is validated before anything is enqueued; on error nothing
 * changes. Errors: those of hs_kv_import (the message names the blob). */
hs_status hs_kv_import_many(hs_stage* st, int32_t n_blobs, const void* const* srcs,
                            const uint64_t* bytes, const void* const* heads,
                            const uint64_t* head_bytes, void* stream);

/* Host-staged (streaming) migration, the form that crosses machines
 * (section 6.2: blocks leave the GPU in chunks that are sent on as soon as
 * they reach host memory, and on the receiving worker each arriving chunk
 * is loaded to the GPU on its own stream). Blobs are the same bytes as
 * above; chunks are whole KV units of about `chunk_bytes` (the first one
 * also carries the header and records).
 *
 * hs_kv_export_host: like hs_kv_export, but `dst` is pinned host memory
 * (hs_host_alloc). The blocks are gathered chunk by chunk into a device
 * staging buffer owned by the stage (grown on demand) and every chunk is
 * copied to `dst` on `stream` as soon as it is gathered.
 * hs_kv_host_progress reports the landed prefix without blocking; the call
 * as a whole is complete (ordered on `stream` and for later calls) when
 * every chunk has landed.
 *
 * hs_kv_import_host: like hs_kv_import, but `src` is a complete blob in
 * pinned host memory. The header is read from host memory; the chunks are
 * copied to the staging buffer on the copy streams and each chunk's units
 * are scattered into the pools (on `stream`) as soon as it has landed.
 *
 * Errors: as hs_kv_export / hs_kv_import; HS_EINVAL also for memory that is
 * not pinned host memory or chunk_bytes == 0; HS_ENOMEM when the staging
 * buffer cannot grow. */
hs_status hs_kv_export_host(hs_stage* st, int32_t n_seqs, const int64_t* seq_ids,
                            void* dst, uint64_t cap, uint64_t chunk_bytes,
                            uint64_t* written, void* stream);
hs_status hs_kv_import_host(hs_stage* st, const void* src, uint64_t bytes,
                            uint64_t chunk_bytes, void* stream);
/* Bytes of the last host-staged transfer that have landed, as a prefix. */
hs_status hs_kv_host_progress(hs_stage* st, uint64_t* landed);

/* Consolidate: `dst` takes over the sequences of the `n_srcs` source stages
 * (section 6.1 scaling down). The serving ranges of dst (if not empty) and
 * of all sources must be disjoint and together contiguous, within dst's
 * resident range, with every needed dst weight chunk submitted. Every
 * source must hold the same live {seq_id, n_tokens} set, and dst either
 * none of them or the same set. The call orders itself after all work of
 * the sources (drain), copies their KV blocks device-to-device into dst at
 * the sources' layers, sets dst's serving range to the union and releases
 * the sequences in the sources. Errors: HS_EINVAL, HS_ESTATE (ranges, sets,
 * missing weights), HS_ENOMEM, HS_EHIP; on error nothing changes. */
hs_status hs_stage_merge(hs_stage* dst, hs_stage* const* srcs, int32_t n_srcs,
                         void* stream);

/* Parse and validate a blob header held in host memory (`avail` bytes of
 * the blob's start, at least 64 + 16 n_seqs). Host-only. */
typedef struct {
  int32_t layer_begin, layer_end, n_kv_heads, head_dim, block_size, n_seqs;
  uint64_t payload_offset, payload_bytes, total_bytes;
} hs_kv_blob_info;

hs_status hs_kv_blob_describe(const void* host_blob, uint64_t avail,
                              hs_kv_blob_info* out);

/* ------------------------------------------------------------------------
 * Measurement. When timing is on, the stage's kernel launches are bracketed
 * by HIP events on their stream: every launch, or only those of the launch
 * sites named by hs_stage_set_timing_sites (a comma-separated list of
 * "embed", "attn_norm", "qkv" (the QKV projection with RoPE and the KV
 * append), "attn", "o_proj", "ffn_norm", "gate_up", "down", "final_norm",
 * "lm_head", "argmax", "kv_copy"; a per-layer site followed by "@<layer>",
 * e.g. "gate_up@12", names that layer's launch only; NULL or
 * "" = every site). Events between back-to-back kernels cost time of their
 * own, so timing a few sites disturbs a step less than timing all of them.
 * hs_stage_read_timing waits for the stage, then reports per (kernel, launch
 * site) pair: launches, total milliseconds and the algorithmic flops and
 * HBM bytes of those launches; and resets the counters. `n` receives the
 * number of pairs, of which min(n, cap) are written.
 */
typedef struct {
  char name[48];
  char site[16];
  int64_t launches;
  double total_ms;
  double flops;
  double bytes;
} hs_kernel_stat;

hs_status hs_stage_set_timing(hs_stage* st, int32_t enable);
hs_status hs_stage_set_timing_sites(hs_stage* st, const char* sites);
hs_status hs_stage_read_timing(hs_stage* st, hs_kernel_stat* out, int32_t cap,
                               int32_t* n);

/* Thread-local description of the last error (never NULL). */
const char* hs_last_error(void);

/* Page-locked host memory (hipHostMalloc) from the HIP runtime the library
 * itself uses, for weight images (hs_stage_load_chunk) and host-staged KV
 * blobs. Memory the GPU copies from or to must be known to that runtime as
 * page-locked: a buffer locked by another runtime instance in the process
 * is copied through staging buffers, at a fraction of the host-link rate.
 * hs_host_free(NULL) is a no-op. Errors: HS_EINVAL (null out), HS_ENOMEM. */
hs_status hs_host_alloc(uint64_t bytes, void** out);
hs_status hs_host_free(void* p);

#ifdef __cplusplus
}
#endif

#endif /* HS_H */
