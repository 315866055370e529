"""Marshalling helpers around the C ABI: model configs, pinned weight images,
chunked loading, and a small owner object for a stage handle.

Nothing here computes any part of the model; every step of the forward pass,
the KV cache and the weight upload runs inside libhs.so.
"""
from __future__ import annotations

import concurrent.futures as cf

import numpy as np

from workloads import gen
from . import hs

NORMS = ("attn_norm", "ffn_norm", "final_norm")
LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wgate", "wup", "wdown")


def hs_cfg(cfg) -> hs.hs_model_cfg:
    """C struct for a ``workloads.ModelCfg``."""
    return hs.model_cfg(cfg.n_layers, cfg.hidden, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                        cfg.ffn, cfg.vocab, cfg.rms_eps, cfg.rope_base)


def image_tensors(cfg, rb, re):
    """(layer, kind) of every tensor in the image of resident layers [rb, re)."""
    out = []
    if rb == 0:
        out.append((-1, "embed"))
    for l in range(rb, re):
        out.extend((l, k) for k in LAYER_TENSORS)
    if re == cfg.n_layers:
        out.extend([(-1, "final_norm"), (-1, "lm_head")])
    return out


def seeded_source(cfg):
    """The seeded float32 draws of ``workloads.gen`` (gains are ones)."""
    def src(layer, kind):
        if kind in NORMS:
            return gen.gains(cfg)
        return gen.weight_f32(cfg, layer, kind)
    return src


def pack_image(cfg, rb, re, image_ptr, source=None, threads=8):
    """Write every tensor of the stage image into host memory at image_ptr,
    as bf16 (round to nearest even) in the library's layout."""
    c = hs_cfg(cfg)
    source = source or seeded_source(cfg)

    def one(item):
        layer, kind = item
        bits = gen.to_bf16_bits(np.asarray(source(layer, kind), dtype=np.float32))
        hs.hs_image_put(c, rb, re, layer, kind, bits.ctypes.data, bits.size, image_ptr)

    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(one, image_tensors(cfg, rb, re)))


class PinnedBuffer:
    """Page-locked host memory from the library (hs_host_alloc, i.e.
    hipHostMalloc in the HIP runtime the library and torch share), released
    on close() or garbage collection (not cached). Exposes data_ptr() and
    numel() (bytes)."""

    def __init__(self, nbytes):
        self._p = hs.hs_host_alloc(nbytes)
        self._n = nbytes

    def data_ptr(self):
        return self._p

    def numel(self):
        return self._n

    def numpy(self):
        import ctypes
        return np.ctypeslib.as_array((ctypes.c_uint8 * self._n).from_address(self._p))

    def close(self):
        if self._p:
            hs.hs_host_free(self._p)
            self._p = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def pinned_image(cfg, rb, re, source=None):
    """A PinnedBuffer holding the packed image of resident layers [rb, re)."""
    _, nbytes = hs.hs_weight_layout(hs_cfg(cfg), rb, re)
    img = PinnedBuffer(nbytes)
    pack_image(cfg, rb, re, img.data_ptr(), source)
    return img


def load_image(h, image, chunk_bytes=32 << 20, order=None):
    """Submit the whole image as chunks (optionally in a given chunk order)."""
    n = image.numel()
    base = image.data_ptr()
    offs = list(range(0, n, chunk_bytes))
    if order is not None:
        offs = [offs[i] for i in order]
    for off in offs:
        hs.hs_stage_load_chunk(h, off, base + off, min(chunk_bytes, n - off))
    return len(offs)


class Stage:
    """Owns one hs_stage handle (destroyed on close / garbage collection)."""

    def __init__(self, cfg, begin, end, max_seqs=8, max_ctx=256, max_batch_tokens=1024,
                 resident=None, kv_num_blocks=0, n_copy_streams=2, device=0):
        self.cfg = cfg
        self.c = hs_cfg(cfg)
        rb, re = resident if resident else (begin, end)
        self.resident = (rb, re)
        self.opts = hs.stage_opts(max_seqs, max_ctx, max_batch_tokens, (rb, re),
                                  kv_num_blocks, n_copy_streams)
        self.h = hs.hs_stage_create(self.c, begin, end, self.opts, device)

    @property
    def begin(self):
        return self.info()["layer_begin"]

    @property
    def end(self):
        return self.info()["layer_end"]

    def close(self):
        if getattr(self, "h", None) is not None:
            hs.hs_stage_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # thin forwards
    def load(self, image, chunk_bytes=32 << 20, order=None):
        return load_image(self.h, image, chunk_bytes, order)

    def prefill(self, ids, lens, inp, out, logits=0, stream=0):
        hs.hs_stage_prefill(self.h, ids, lens, inp, out, logits, stream)

    def decode(self, ids, inp, out, logits=0, stream=0):
        hs.hs_stage_decode(self.h, ids, inp, out, logits, stream)

    def sync(self):
        hs.hs_stage_sync(self.h)

    def info(self):
        return hs.hs_stage_get_info(self.h)
