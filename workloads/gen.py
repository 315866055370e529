"""Seeded generators for weights, prompts and stage inputs.

Every tensor has its own counter-seeded stream, ``default_rng([0, layer + 1,
tensor_id])``, with ``layer + 1 = 0`` for the embedding, the final norm and the
LM head. A stage can therefore draw exactly its own layers, and the oracle and
the engine see the same numbers without either one producing the other's
inputs. Matrices and the embedding are N(0, 0.02) in float32; RMSNorm gains
are 1.0. The engine stores weights in bfloat16, rounded to nearest-even from
the same float32 draw.
"""
from __future__ import annotations

import numpy as np

# Tensor ids used in the per-tensor seed.
TENSOR_IDS = {
    "embed": 0, "wq": 1, "wk": 2, "wv": 3, "wo": 4,
    "wgate": 5, "wup": 6, "wdown": 7, "lm_head": 8,
}

WEIGHT_STD = 0.02


def weight_shape(cfg, kind: str):
    h, f = cfg.hidden, cfg.ffn
    return {
        "embed": (cfg.vocab, h),
        "wq": (cfg.q_dim, h),
        "wk": (cfg.kv_dim, h),
        "wv": (cfg.kv_dim, h),
        "wo": (h, cfg.q_dim),
        "wgate": (f, h),
        "wup": (f, h),
        "wdown": (h, f),
        "lm_head": (cfg.vocab, h),
    }[kind]


def weight_f32(cfg, layer: int, kind: str) -> np.ndarray:
    """float32 draw of one weight matrix; ``layer`` is ignored for the
    embedding and LM head (their seed uses layer slot 0)."""
    tid = TENSOR_IDS[kind]
    slot = 0 if kind in ("embed", "lm_head") else layer + 1
    rng = np.random.default_rng([0, slot, tid])
    w = rng.standard_normal(weight_shape(cfg, kind), dtype=np.float32)
    w *= np.float32(WEIGHT_STD)
    return w


def gains(cfg) -> np.ndarray:
    """RMSNorm gains (attention, FFN and final norms): all ones."""
    return np.ones(cfg.hidden, dtype=np.float32)


def tokens(vocab: int, n: int, seed: int) -> np.ndarray:
    """``n`` uniform token ids in [0, vocab) from stream [1, seed]."""
    rng = np.random.default_rng([1, seed])
    return rng.integers(0, vocab, n).astype(np.int32)


def ragged_lengths(lo: int, hi_inclusive: int, n: int, seed: int):
    rng = np.random.default_rng(seed)
    return [int(x) for x in rng.integers(lo, hi_inclusive + 1, n)]


def hidden_input(n_tokens: int, hidden: int, seed: int) -> np.ndarray:
    """A synthetic float32 residual-stream input for a middle stage, of unit
    scale, from stream [2, seed]."""
    rng = np.random.default_rng([2, seed])
    return rng.standard_normal((n_tokens, hidden), dtype=np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite value in bf16 conversion")
    u = x.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16, returned as float32."""
    return bf16_bits_to_f32(to_bf16_bits(x))
