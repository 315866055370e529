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
