"""Independent codec for the KV export blob. TEST INFRASTRUCTURE ONLY.

The paper (section 6.2) moves the cache blocks of every unfinished request
from the stage workers to the worker that holds the whole model, where they
are placed at the layers of the worker they came from. It does not define a
wire format. The engine's blob is self-describing, little-endian:

  offset  size  field
  0       4     magic b"HSKV"
  4       4     u32 version (1)
  8       4     u32 dtype (1 = bfloat16)
  12      4     i32 layer_begin
  16      4     i32 layer_end          (the layers the payload covers)
  20      4     i32 n_kv_heads
  24      4     i32 head_dim
  28      4     i32 block_size         (tokens per block)
  32      4     i32 n_seqs
  36      4     u32 reserved (0)
  40      8     u64 payload_offset = align_up(64 + 16 * n_seqs, 256)
  48      8     u64 payload_bytes
  56      8     u64 total_bytes    = payload_offset + payload_bytes
  64      16*n  per sequence: i64 seq_id, i32 n_tokens, i32 n_blocks
                (n_blocks = ceil(n_tokens / block_size)); zero padding up to
                payload_offset
  payload: for each layer, for each sequence in record order, for each of
           its blocks: the K block [n_kv][block_size][head_dim] then the V
           block, bfloat16; token slots past n_tokens are zero.

This module packs and parses that format from its description only; it does
not share code with the engine's C++ codec.
"""
from __future__ import annotations

import struct

import numpy as np

MAGIC = b"HSKV"
VERSION = 1
DTYPE_BF16 = 1
HEADER = struct.Struct("<4sIIiiiiiiIQQQ")
RECORD = struct.Struct("<qii")
assert HEADER.size == 64 and RECORD.size == 16


def _align(n, a):
    return (n + a - 1) // a * a


def blob_size(n_layers, n_kv, head_dim, block_size, n_tokens_list):
    nblk = sum(-(-n // block_size) for n in n_tokens_list)
    payload = n_layers * nblk * 2 * n_kv * block_size * head_dim * 2
    return _align(64 + 16 * len(n_tokens_list), 256) + payload


def pack(layer_begin, layer_end, n_kv, head_dim, block_size, seqs):
    """seqs: list of (seq_id, K, V) with K, V uint16 bfloat16 bit patterns of
    shape [layer_end - layer_begin, n_tokens, n_kv, head_dim]."""
    n_layers = layer_end - layer_begin
    recs = []
    for sid, k, v in seqs:
        assert k.shape == v.shape and k.shape[0] == n_layers
        assert k.shape[2] == n_kv and k.shape[3] == head_dim
        n = k.shape[1]
        recs.append((sid, n, -(-n // block_size)))
    poff = _align(64 + 16 * len(recs), 256)
    blk_elems = n_kv * block_size * head_dim
    payload = np.zeros(n_layers * sum(r[2] for r in recs) * 2 * blk_elems,
                       dtype=np.uint16)
    pos = 0
    for li in range(n_layers):
        for (sid, n, nb), (_, k, v) in zip(recs, seqs):
            for b in range(nb):
                for src in (k, v):
                    blk = np.zeros((n_kv, block_size, head_dim), np.uint16)
                    t0, t1 = b * block_size, min(n, (b + 1) * block_size)
                    # token-major [tok][head][d] -> block [head][slot][d]
                    blk[:, :t1 - t0, :] = np.transpose(src[li, t0:t1], (1, 0, 2))
                    payload[pos:pos + blk_elems] = blk.reshape(-1)
                    pos += blk_elems
    pbytes = payload.nbytes
    hdr = HEADER.pack(MAGIC, VERSION, DTYPE_BF16, layer_begin, layer_end,
                      n_kv, head_dim, block_size, len(recs), 0, poff, pbytes,
                      poff + pbytes)
    body = b"".join(RECORD.pack(*r) for r in recs)
    pad = b"\0" * (poff - 64 - len(body))
    return hdr + body + pad + payload.tobytes()


def parse(blob):
    """Inverse of ``pack``: returns (header dict, list of (seq_id, K, V))."""
    blob = bytes(blob)
    (magic, ver, dt, lb, le, n_kv, d, bs, n, _r, poff, pbytes,
     total) = HEADER.unpack_from(blob, 0)
    if magic != MAGIC or ver != VERSION or dt != DTYPE_BF16:
        raise ValueError("not a v1 bf16 KV blob")
    if total != len(blob) or poff + pbytes != total:
        raise ValueError("size fields disagree with the blob length")
    recs = [RECORD.unpack_from(blob, 64 + 16 * i) for i in range(n)]
    n_layers = le - lb
    blk_elems = n_kv * bs * d
    payload = np.frombuffer(blob, dtype=np.uint16, offset=poff)
    out = [(sid, np.zeros((n_layers, nt, n_kv, d), np.uint16),
            np.zeros((n_layers, nt, n_kv, d), np.uint16)) for sid, nt, _ in recs]
    pos = 0
    for li in range(n_layers):
        for (sid, nt, nb), (_, k, v) in zip(recs, out):
            for b in range(nb):
                for dst in (k, v):
                    blk = payload[pos:pos + blk_elems].reshape(n_kv, bs, d)
                    t0, t1 = b * bs, min(nt, (b + 1) * bs)
                    dst[li, t0:t1] = np.transpose(blk[:, :t1 - t0, :], (1, 0, 2))
                    pos += blk_elems
    hdr = dict(layer_begin=lb, layer_end=le, n_kv_heads=n_kv, head_dim=d,
               block_size=bs, n_seqs=n, payload_offset=poff,
               payload_bytes=pbytes, total_bytes=total,
               records=[(sid, nt, nb) for sid, nt, nb in recs])
    return hdr, out
