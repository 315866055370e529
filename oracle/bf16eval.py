"""The decoder evaluated with 16-bit storage: the oracle's arithmetic with
every stored tensor rounded to bfloat16. TEST INFRASTRUCTURE ONLY.

Purpose: a tolerance for comparing a bf16 engine with the float32 oracle
over many layers. Section 8 of the paper serves its models in 16-bit floats,
and section 4.1 prices the stage boundary at one 16-bit hidden vector per
token (8 KB at hidden size 4096); an implementation that stores weights and
activations in 16 bits therefore differs from the float32 definition by the
rounding of what it stores, and that difference grows with depth. This
module measures it on the CPU: the float32 oracle's steps, unchanged, with a
round-to-nearest-even bfloat16 rounding applied to

* every weight matrix and the embedding rows,
* the normalised activation entering each projection,
* q, k and v as projected, and q and k again after the rotation,
* the attention output,
* the residual stream after each of the two residual additions (the sum is
  formed in float32 and rounded once),
* the SwiGLU product silu(gate) * up (formed from float32 gate and up),

while the logits are not rounded. Arithmetic is float32 like the oracle's (or
float64 on request, to see how much the accumulation order matters). These are the storage points of the engine's
bfloat16 residual-stream design (bf16 storage, float32 accumulation, float32
norms and softmax). Everything else, including the order of operations, is
the oracle's. With ``rounding=False`` the evaluation is the float32 oracle
itself, bit for bit (pinned in ``tests/test_bf16_budget.py``).
"""
from __future__ import annotations

import numpy as np

from workloads import gen as _gen

from .llama import Stage, apply_rope, attention, rms_norm, rope_angles, silu


class Bf16Stage(Stage):
    """``oracle.llama.Stage`` with the bfloat16 storage described above.

    Takes the same float32 weight source as ``Stage``; weights are rounded
    when read. The KV cache holds the rounded, rotated keys and the rounded
    values."""

    def __init__(self, cfg, weights, begin, end, rounding=True, dtype=np.float32):
        super().__init__(cfg, weights, begin, end, dtype)
        self.rounding = rounding

    def _r(self, a):
        """Round to bfloat16 (via float32), kept in the arithmetic dtype."""
        if not self.rounding:
            return np.asarray(a, dtype=self.dtype)
        return _gen.round_to_bf16(np.asarray(a, dtype=np.float32)).astype(self.dtype)

    def _w(self, layer, kind):
        w = np.asarray(self.W(layer, kind), dtype=np.float32)
        if kind in ("attn_norm", "ffn_norm", "final_norm"):
            return w.astype(self.dtype)     # gains are 1.0, exact in bf16
        return self._r(w)

    def _layer(self, l, x, pos, seq_id):
        cfg, r = self.cfg, self._r
        n = x.shape[0]
        u = r(rms_norm(x, self._w(l, "attn_norm"), cfg.rms_eps))
        q = r(u @ self._w(l, "wq").T).reshape(n, cfg.n_heads, cfg.head_dim)
        k = r(u @ self._w(l, "wk").T).reshape(n, cfg.n_kv_heads, cfg.head_dim)
        v = r(u @ self._w(l, "wv").T).reshape(n, cfg.n_kv_heads, cfg.head_dim)
        cos, sin = rope_angles(pos, cfg.head_dim, cfg.rope_base)
        q = r(apply_rope(q, cos, sin))
        k = r(apply_rope(k, cos, sin))
        cache = self.kv.setdefault(seq_id, {})
        if l in cache:
            k_all = np.concatenate([cache[l][0], k], axis=0)
            v_all = np.concatenate([cache[l][1], v], axis=0)
        else:
            k_all, v_all = k, v
        cache[l] = (k_all, v_all)
        o = r(attention(q, k_all, v_all, pos, np.arange(k_all.shape[0])))
        x = r(x + o @ self._w(l, "wo").T)
        u = r(rms_norm(x, self._w(l, "ffn_norm"), cfg.rms_eps))
        a = r(silu(u @ self._w(l, "wgate").T) * (u @ self._w(l, "wup").T))
        return r(x + a @ self._w(l, "wdown").T)

    def _run(self, seq_id, inp, pos):
        cfg = self.cfg
        if self.begin == 0:
            x = self._w(-1, "embed")[np.asarray(inp, dtype=np.int64)]
        else:
            x = self._r(inp)
        for l in range(self.begin, self.end):
            x = self._layer(l, x, pos, seq_id)
        if self.end == cfg.n_layers:
            u = self._r(rms_norm(x, self._w(-1, "final_norm"), cfg.rms_eps))
            return u @ self._w(-1, "lm_head").T
        return x


def logit_err(got, ref):
    """max |got - ref| / max |ref| over the last axis' rows (worst row)."""
    got = np.atleast_2d(np.asarray(got, np.float64))
    ref = np.atleast_2d(np.asarray(ref, np.float64))
    return float(np.max(np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)))


def hidden_err(got, ref):
    """Relative Frobenius error of hidden states."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
