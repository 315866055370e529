"""ctypes binding of the C ABI in include/hs.h.

Functions keep the C names and only marshal arguments: pointers are passed
as Python ints (e.g. ``tensor.data_ptr()``), host id/length lists as Python
sequences, streams as ``torch.cuda.Stream.cuda_stream`` ints (0 = the null
stream, which is torch's default stream). Failures raise ``HSError`` carrying the status and the
library's message. All work runs in libhs.so; if the library has not been
built, every call raises.
"""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libhs.so")

HS_OK, HS_EINVAL, HS_ENOMEM, HS_ENOTREADY, HS_ERANGE, HS_ESTATE, HS_EHIP = 0, -1, -2, -3, -4, -5, -6
STATUS_NAMES = {0: "HS_OK", -1: "HS_EINVAL", -2: "HS_ENOMEM", -3: "HS_ENOTREADY",
                -4: "HS_ERANGE", -5: "HS_ESTATE", -6: "HS_EHIP"}

# weight kinds in the image
(HS_W_EMBED, HS_W_ATTN_NORM, HS_W_QKV, HS_W_O, HS_W_FFN_NORM, HS_W_GATEUP, HS_W_DOWN,
 HS_W_FINAL_NORM, HS_W_LM_HEAD) = range(9)
# standard source tensors for hs_image_put
SRC_KINDS = {"embed": 0, "attn_norm": 1, "wq": 2, "wk": 3, "wv": 4, "wo": 5, "ffn_norm": 6,
             "wgate": 7, "wup": 8, "wdown": 9, "final_norm": 10, "lm_head": 11}


class HSError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class hs_model_cfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_float), ("rope_base", C.c_float)]


class hs_stage_opts(C.Structure):
    _fields_ = [("resident_begin", C.c_int32), ("resident_end", C.c_int32),
                ("max_seqs", C.c_int32), ("max_ctx", C.c_int32),
                ("max_batch_tokens", C.c_int32), ("kv_block_size", C.c_int32),
                ("kv_num_blocks", C.c_int32), ("n_copy_streams", C.c_int32)]


class hs_tensor_desc(C.Structure):
    _fields_ = [("offset", C.c_uint64), ("bytes", C.c_uint64), ("layer", C.c_int32),
                ("kind", C.c_int32), ("rows", C.c_int64), ("cols", C.c_int64),
                ("tiled", C.c_int32), ("reserved", C.c_int32)]


class hs_stage_info(C.Structure):
    _fields_ = [("layer_begin", C.c_int32), ("layer_end", C.c_int32),
                ("resident_begin", C.c_int32), ("resident_end", C.c_int32),
                ("live_seqs", C.c_int32), ("free_blocks", C.c_int32),
                ("total_blocks", C.c_int32), ("block_size", C.c_int32),
                ("image_bytes", C.c_uint64), ("kv_bytes", C.c_uint64)]


class hs_kv_blob_info(C.Structure):
    _fields_ = [("layer_begin", C.c_int32), ("layer_end", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("block_size", C.c_int32), ("n_seqs", C.c_int32),
                ("payload_offset", C.c_uint64), ("payload_bytes", C.c_uint64),
                ("total_bytes", C.c_uint64)]


class hs_kernel_stat(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("site", C.c_char * 16), ("launches", C.c_int64),
                ("total_ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_P = C.c_void_p
_SIGS = {
    "hs_weight_layout": [C.POINTER(hs_model_cfg), C.c_int32, C.c_int32,
                         C.POINTER(hs_tensor_desc), C.c_int32, C.POINTER(C.c_int32),
                         C.POINTER(C.c_uint64)],
    "hs_image_put": [C.POINTER(hs_model_cfg), C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                     _P, C.c_uint64, _P],
    "hs_stage_create": [C.POINTER(hs_model_cfg), C.c_int32, C.c_int32,
                        C.POINTER(hs_stage_opts), C.c_int32, C.POINTER(_P)],
    "hs_stage_destroy": [_P],
    "hs_stage_sync": [_P],
    "hs_stage_load_chunk": [_P, C.c_uint64, _P, C.c_uint64],
    "hs_stage_loaded": [_P, C.POINTER(C.c_int32), C.POINTER(C.c_uint64)],
    "hs_stage_invalidate_weights": [_P],
    "hs_stage_prefill": [_P, C.c_int32, C.POINTER(C.c_int64), C.POINTER(C.c_int32), _P, _P,
                         _P, _P],
    "hs_stage_decode": [_P, C.c_int32, C.POINTER(C.c_int64), _P, _P, _P, _P],
    "hs_seq_free": [_P, C.c_int64],
    "hs_seq_tokens": [_P, C.c_int64, C.POINTER(C.c_int32)],
    "hs_stage_get_info": [_P, C.POINTER(hs_stage_info)],
    "hs_kv_export_size": [_P, C.c_int32, C.POINTER(C.c_int64), C.POINTER(C.c_uint64)],
    "hs_kv_export": [_P, C.c_int32, C.POINTER(C.c_int64), _P, C.c_uint64,
                     C.POINTER(C.c_uint64), _P],
    "hs_kv_import": [_P, _P, C.c_uint64, _P],
    "hs_host_alloc": [C.c_uint64, C.POINTER(_P)],
    "hs_host_free": [_P],
    "hs_kv_export_head": [_P, C.c_int32, C.POINTER(C.c_int64), _P, C.c_uint64,
                          C.POINTER(C.c_uint64)],
    "hs_kv_import_many": [_P, C.c_int32, C.POINTER(_P), C.POINTER(C.c_uint64), C.POINTER(_P),
                          C.POINTER(C.c_uint64), _P],
    "hs_kv_export_host": [_P, C.c_int32, C.POINTER(C.c_int64), _P, C.c_uint64, C.c_uint64,
                          C.POINTER(C.c_uint64), _P],
    "hs_kv_import_host": [_P, _P, C.c_uint64, C.c_uint64, _P],
    "hs_kv_host_progress": [_P, C.POINTER(C.c_uint64)],
    "hs_stage_merge": [_P, C.POINTER(_P), C.c_int32, _P],
    "hs_kv_blob_describe": [_P, C.c_uint64, C.POINTER(hs_kv_blob_info)],
    "hs_stage_set_timing": [_P, C.c_int32],
    "hs_stage_set_timing_sites": [_P, C.c_char_p],
    "hs_stage_read_timing": [_P, C.POINTER(hs_kernel_stat), C.c_int32, C.POINTER(C.c_int32)],
    # single-kernel entry points (include/hs_kernel.h)
    "hs_k_gemm": [_P, C.c_int64, _P, _P, C.c_int64, _P, C.c_int64, C.c_int32, C.c_int32,
                  C.c_int32, C.c_int32, _P],
    "hs_pack_tiled": [_P, C.c_int64, C.c_int64, _P],
    "hs_k_attn_prefill": [_P, _P, C.POINTER(C.c_int32), C.c_int32, C.c_int32, C.c_int32,
                          C.c_int32, _P],
    "hs_k_gemm_rmsnorm": [_P, C.c_int64, _P, C.c_float, _P, _P, C.c_int64, _P, C.c_int64,
                          C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P],
    "hs_k_rmsnorm": [_P, _P, _P, C.c_int32, C.c_int32, C.c_float, _P],
    "hs_k_attn_decode": [_P, C.c_int64, _P, _P, _P, _P, C.c_int64, C.c_int32, C.c_int32,
                         C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P],
    "hs_k_attn_decode_noalloc": [_P, C.c_int64, _P, _P, _P, _P, C.c_int64, C.c_int32,
                                 C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _P],
    "hs_k_argmax": [_P, C.c_int32, C.c_int32, _P, _P],
    "hs_k_attn_decode_rope": [_P, C.c_int64, _P, _P, _P, _P, _P, C.c_int32, _P, C.c_int64,
                              C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                              _P],
}
EXPORTED = sorted(list(_SIGS) + ["hs_last_error"])

_lib = None


def lib():
    """Load libhs.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise HSError(HS_EINVAL, f"{LIB_PATH} is missing; build it with "
                          "`python -m paper_2502_15524_amd.build`")
        # torch ships its own HIP runtime under the same soname as the one
        # libhs.so links against. Loaded first, torch's copy is the one both
        # use; loaded the other way round, the process ends up with two
        # runtimes and the library's sees no device. So torch goes first.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        l = C.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            f = getattr(l, name)
            f.argtypes = args
            f.restype = C.c_int
        l.hs_last_error.argtypes = []
        l.hs_last_error.restype = C.c_char_p
        _lib = l
    return _lib


def hs_last_error() -> str:
    return lib().hs_last_error().decode()


def _check(code):
    if code != HS_OK:
        raise HSError(code, hs_last_error())


def _i64(seq):
    seq = [int(x) for x in seq]
    return (C.c_int64 * len(seq))(*seq), len(seq)


def _i32(seq):
    seq = [int(x) for x in seq]
    return (C.c_int32 * len(seq))(*seq)


def model_cfg(n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab, rms_eps=1e-5,
              rope_base=10000.0) -> hs_model_cfg:
    return hs_model_cfg(n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab, rms_eps,
                        rope_base)


def stage_opts(max_seqs, max_ctx, max_batch_tokens, resident=(0, 0), kv_num_blocks=0,
               n_copy_streams=2, kv_block_size=16) -> hs_stage_opts:
    return hs_stage_opts(resident[0], resident[1], max_seqs, max_ctx, max_batch_tokens,
                         kv_block_size, kv_num_blocks, n_copy_streams)


# ----------------------------------------------------------------- host-only

def hs_weight_layout(cfg, resident_begin, resident_end):
    n = C.c_int32(0)
    nbytes = C.c_uint64(0)
    _check(lib().hs_weight_layout(C.byref(cfg), resident_begin, resident_end, None, 0,
                                  C.byref(n), C.byref(nbytes)))
    arr = (hs_tensor_desc * n.value)()
    _check(lib().hs_weight_layout(C.byref(cfg), resident_begin, resident_end, arr, n.value,
                                  C.byref(n), C.byref(nbytes)))
    descs = [dict(offset=d.offset, bytes=d.bytes, layer=d.layer, kind=d.kind, rows=d.rows,
                  cols=d.cols, tiled=d.tiled) for d in arr]
    return descs, nbytes.value


def hs_image_put(cfg, resident_begin, resident_end, layer, src_kind, src_ptr, n_elems,
                 image_ptr):
    if isinstance(src_kind, str):
        src_kind = SRC_KINDS[src_kind]
    _check(lib().hs_image_put(C.byref(cfg), resident_begin, resident_end, layer, src_kind,
                              src_ptr, n_elems, image_ptr))


def hs_kv_blob_describe(blob_head: bytes):
    info = hs_kv_blob_info()
    buf = C.create_string_buffer(bytes(blob_head), len(blob_head))
    _check(lib().hs_kv_blob_describe(buf, len(blob_head), C.byref(info)))
    return {k: getattr(info, k) for k, _ in hs_kv_blob_info._fields_}


# ------------------------------------------------------------------- stages

def hs_stage_create(cfg, layer_begin, layer_end, opts, device=0):
    h = _P()
    _check(lib().hs_stage_create(C.byref(cfg), layer_begin, layer_end, C.byref(opts), device,
                                 C.byref(h)))
    return h


def hs_stage_destroy(h):
    _check(lib().hs_stage_destroy(h))


def hs_stage_sync(h):
    _check(lib().hs_stage_sync(h))


def hs_stage_load_chunk(h, image_offset, src_ptr, nbytes):
    _check(lib().hs_stage_load_chunk(h, image_offset, src_ptr, nbytes))


def hs_stage_loaded(h):
    n = C.c_int32(0)
    w = C.c_uint64(0)
    _check(lib().hs_stage_loaded(h, C.byref(n), C.byref(w)))
    return n.value, w.value


def hs_stage_invalidate_weights(h):
    _check(lib().hs_stage_invalidate_weights(h))


def hs_stage_prefill(h, seq_ids, seq_lens, in_ptr, out_ptr, logits_ptr=0, stream=0):
    ids, n = _i64(seq_ids)
    _check(lib().hs_stage_prefill(h, n, ids, _i32(seq_lens), in_ptr, out_ptr, logits_ptr or None,
                                  stream or None))


def hs_stage_decode(h, seq_ids, in_ptr, out_ptr, logits_ptr=0, stream=0):
    ids, n = _i64(seq_ids)
    _check(lib().hs_stage_decode(h, n, ids, in_ptr, out_ptr, logits_ptr or None,
                                 stream or None))


def hs_seq_free(h, seq_id):
    _check(lib().hs_seq_free(h, seq_id))


def hs_seq_tokens(h, seq_id):
    n = C.c_int32(0)
    _check(lib().hs_seq_tokens(h, seq_id, C.byref(n)))
    return n.value


def hs_stage_get_info(h):
    i = hs_stage_info()
    _check(lib().hs_stage_get_info(h, C.byref(i)))
    return {k: getattr(i, k) for k, _ in hs_stage_info._fields_}


def hs_kv_export_size(h, seq_ids):
    ids, n = _i64(seq_ids)
    b = C.c_uint64(0)
    _check(lib().hs_kv_export_size(h, n, ids, C.byref(b)))
    return b.value


def hs_kv_export(h, seq_ids, dst_ptr, cap, stream=0):
    ids, n = _i64(seq_ids)
    w = C.c_uint64(0)
    code = lib().hs_kv_export(h, n, ids, dst_ptr, cap, C.byref(w), stream or None)
    if code == HS_ERANGE:
        err = HSError(code, hs_last_error())
        err.required = w.value
        raise err
    _check(code)
    return w.value


def hs_kv_import(h, src_ptr, nbytes, stream=0):
    _check(lib().hs_kv_import(h, src_ptr, nbytes, stream or None))


def hs_host_alloc(nbytes):
    """Page-locked host memory from the library's HIP runtime; returns the
    address (free it with hs_host_free)."""
    p = C.c_void_p()
    _check(lib().hs_host_alloc(nbytes, C.byref(p)))
    return p.value


def hs_host_free(ptr):
    _check(lib().hs_host_free(ptr))


def hs_kv_export_head(h, seq_ids):
    """The header + records (+ padding) of the blob hs_kv_export would write
    for these sequences, as bytes (host)."""
    ids, n = _i64(seq_ids)
    w = C.c_uint64(0)
    code = lib().hs_kv_export_head(h, n, ids, None, 0, C.byref(w))
    if code != HS_ERANGE:
        _check(code)
    buf = C.create_string_buffer(w.value)
    _check(lib().hs_kv_export_head(h, n, ids, buf, w.value, C.byref(w)))
    return buf.raw[:w.value]


def hs_kv_import_many(h, blobs, stream=0):
    """blobs: list of (device pointer, size, head bytes) imported in one
    launch, in order."""
    n = len(blobs)
    srcs = (C.c_void_p * n)(*[b[0] for b in blobs])
    sizes = (C.c_uint64 * n)(*[b[1] for b in blobs])
    keep = [C.create_string_buffer(bytes(b[2]), len(b[2])) for b in blobs]
    heads = (C.c_void_p * n)(*[C.addressof(k) for k in keep])
    hlen = (C.c_uint64 * n)(*[len(b[2]) for b in blobs])
    _check(lib().hs_kv_import_many(h, n, srcs, sizes, heads, hlen, stream or None))


def hs_kv_export_host(h, seq_ids, host_dst, cap, chunk_bytes=64 << 20, stream=0):
    """Export into pinned host memory in chunks; returns the blob size."""
    ids, n = _i64(seq_ids)
    w = C.c_uint64(0)
    code = lib().hs_kv_export_host(h, n, ids, host_dst, cap, chunk_bytes, C.byref(w),
                                   stream or None)
    if code == HS_ERANGE:
        err = HSError(code, hs_last_error())
        err.required = w.value
        raise err
    _check(code)
    return w.value


def hs_kv_import_host(h, host_src, nbytes, chunk_bytes=64 << 20, stream=0):
    _check(lib().hs_kv_import_host(h, host_src, nbytes, chunk_bytes, stream or None))


def hs_kv_host_progress(h):
    v = C.c_uint64(0)
    _check(lib().hs_kv_host_progress(h, C.byref(v)))
    return v.value


def hs_stage_merge(dst, srcs, stream=0):
    arr = (_P * len(srcs))(*[s.value if isinstance(s, _P) else s for s in srcs])
    _check(lib().hs_stage_merge(dst, arr, len(srcs), stream or None))


def hs_stage_set_timing(h, enable):
    _check(lib().hs_stage_set_timing(h, 1 if enable else 0))


def hs_stage_set_timing_sites(h, sites=None):
    """Restrict timing to the named launch sites (list or comma string; None = all)."""
    if sites is not None and not isinstance(sites, str):
        sites = ",".join(sites)
    _check(lib().hs_stage_set_timing_sites(h, sites.encode() if sites else None))


def hs_stage_read_timing(h, cap=256):
    """Per-kernel timing since the last read (waits for the stage; resets)."""
    arr = (hs_kernel_stat * cap)()
    n = C.c_int32(0)
    _check(lib().hs_stage_read_timing(h, arr, cap, C.byref(n)))
    return [dict(name=a.name.decode(), site=a.site.decode(), launches=a.launches,
                 total_ms=a.total_ms,
                 flops=a.flops, bytes=a.bytes) for a in arr[:min(n.value, cap)]]


# ------------------------------------------------------- single kernels

EPI = {"store": 0, "resid": 1, "swiglu": 2, "f32": 3}


def hs_k_gemm(X, ldx, W, Y, ldy, R, ldr, M, N, K, epi, stream=0):
    if isinstance(epi, str):
        epi = EPI[epi]
    _check(lib().hs_k_gemm(X, ldx, W, Y, ldy, R or None, ldr, M, N, K, epi, stream or None))


def hs_k_gemm_rmsnorm(X, ldx, g, eps, W, Y, ldy, R, ldr, M, N, K, epi, stream=0):
    if isinstance(epi, str):
        epi = EPI[epi]
    _check(lib().hs_k_gemm_rmsnorm(X, ldx, g, eps, W, Y, ldy, R or None, ldr, M, N, K, epi,
                                   stream or None))


def hs_pack_tiled(src_ptr, rows, cols, dst_ptr):
    """Row-major bf16 [rows][cols] at src_ptr -> tiled matrix format at dst_ptr."""
    _check(lib().hs_pack_tiled(src_ptr, rows, cols, dst_ptr))


def hs_k_attn_prefill(qkv, out, cu_seqlens, n_heads, n_kv_heads, head_dim, stream=0):
    cu = _i32(cu_seqlens)
    _check(lib().hs_k_attn_prefill(qkv, out, cu, len(cu_seqlens) - 1, n_heads, n_kv_heads,
                                   head_dim, stream or None))


def hs_k_attn_decode(q, ldq, pool, block_table, ctx, out, ldo, B, n_heads, n_kv_heads,
                     head_dim, max_blocks, max_ctx, stream=0):
    """Decode attention over a paged KV pool; block_table and ctx are device pointers."""
    _check(lib().hs_k_attn_decode(q, ldq, pool, block_table, ctx, out, ldo, B, n_heads,
                                  n_kv_heads, head_dim, max_blocks, max_ctx, stream or None))


def hs_k_attn_decode_noalloc(q, ldq, pool, block_table, ctx, out, ldo, B, n_heads, n_kv_heads,
                             head_dim, max_blocks, max_ctx, stream=0):
    """hs_k_attn_decode with its split partials in the library's static
    per-GPU array (no device allocation); calls on one GPU must not overlap."""
    _check(lib().hs_k_attn_decode_noalloc(q, ldq, pool, block_table, ctx, out, ldo, B, n_heads,
                                          n_kv_heads, head_dim, max_blocks, max_ctx,
                                          stream or None))


def hs_k_argmax(logits, n_rows, n_cols, out, stream=0):
    """Greedy token per row: lowest index of the row's maximum (device pointers)."""
    _check(lib().hs_k_argmax(logits, n_rows, n_cols, out, stream or None))


def hs_k_attn_decode_rope(qkv, ldqkv, pool, block_table, ctx, cos_t, sin_t, max_pos, out, ldo,
                          B, n_heads, n_kv_heads, head_dim, max_blocks, max_ctx, stream=0):
    """Decode attention with the step's RoPE and cache append folded in: qkv
    holds the new tokens' projections before RoPE; the rotated key and the
    value are written into the pool slot of position ctx - 1."""
    _check(lib().hs_k_attn_decode_rope(qkv, ldqkv, pool, block_table, ctx, cos_t, sin_t,
                                       max_pos, out, ldo, B, n_heads, n_kv_heads, head_dim,
                                       max_blocks, max_ctx, stream or None))


def hs_k_rmsnorm(x, g, out, rows, hidden, eps, stream=0):
    _check(lib().hs_k_rmsnorm(x, g, out, rows, hidden, eps, stream or None))
