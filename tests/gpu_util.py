"""Helpers shared by the GPU tests: device buffers of bf16 bit patterns and
stage pipelines built from the seeded workloads."""
from __future__ import annotations

import numpy as np

from workloads import gen


def torch():
    import torch as t
    return t


def to_dev_bf16(a):
    """float array -> device torch.bfloat16 tensor (round to nearest even)."""
    t = torch()
    bits = gen.to_bf16_bits(np.asarray(a, dtype=np.float32))
    return t.from_numpy(bits.view(np.int16).copy()).view(t.bfloat16).cuda()


def from_dev_bf16(x):
    t = torch()
    bits = x.contiguous().view(t.int16).cpu().numpy().view(np.uint16)
    return gen.bf16_bits_to_f32(bits)


def stream_ptr():
    return torch().cuda.current_stream().cuda_stream


def rel_fro(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def tiled_index(rows, cols):
    """uint16 element index, in the tiled matrix format, of every (row, col) of
    a [rows][cols] matrix (format: 1 KiB blocks of 8 rows x 64 columns, column
    blocks outermost, chunk c of block row r stored at position c ^ r)."""
    r = np.arange(rows)[:, None]
    c = np.arange(cols)[None, :]
    kb, nb, rr, ch = c // 64, r // 8, r % 8, (c % 64) // 8
    byte = (kb * (rows // 8) + nb) * 1024 + rr * 128 + (ch ^ rr) * 16 + (c % 8) * 2
    return byte // 2


def tile_bits(bits):
    """Row-major uint16 [rows][cols] -> flat tiled uint16 array (zero padded)."""
    rows, cols = bits.shape
    kp = -(-cols // 64) * 64
    out = np.zeros(rows * kp, np.uint16)
    out[tiled_index(rows, cols)] = bits
    return out


def untile_bits(flat, rows, cols):
    return np.asarray(flat)[tiled_index(rows, cols)]
