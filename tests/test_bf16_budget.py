"""The bf16 error budget behind the full-size tolerances (CPU only).

An exact bf16 evaluation of one decoder layer of the 7B shape -- weights and
the activations the engine stores (normed input, q/k/v, rotated q/k, attention
output, residual, SwiGLU output) rounded to bf16, everything else in float64
-- is compared with the float32 oracle. Layer 0 fed from the embedding is the
worst case: its output is all new content, so the rounding is not diluted by
an exactly shared residual. Its error exceeds 1% on its own, which is why the
per-layer hidden-state bound of the full-size GPU tests is 2e-2 and not 1e-2.
"""
import numpy as np

from oracle.llama import Stage, apply_rope, attention, rms_norm, rope_angles, silu
from workloads import MODELS, gen


def test_one_bf16_layer_from_embedding_exceeds_one_percent():
    cfg = MODELS["llama2-7b"]
    T = 128
    rb = gen.round_to_bf16
    W = {k: gen.weight_f32(cfg, 0, k) for k in ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")}
    E = gen.weight_f32(cfg, -1, "embed")
    toks = gen.tokens(cfg.vocab, T, 3)

    def src(layer, kind):
        if kind in ("attn_norm", "ffn_norm", "final_norm"):
            return gen.gains(cfg)
        return E if kind == "embed" else W[kind]

    ref = Stage(MODELS["llama2-7b"], src, 0, 1).prefill([0], [T], toks)

    def f(a):
        return rb(np.asarray(a, np.float32)).astype(np.float64)

    w = {k: rb(v).astype(np.float64) for k, v in W.items()}
    x = rb(E)[toks].astype(np.float64)
    pos = np.arange(T)
    u = f(rms_norm(x, 1.0, cfg.rms_eps))
    q = f(u @ w["wq"].T).reshape(T, cfg.n_heads, cfg.head_dim)
    k = f(u @ w["wk"].T).reshape(T, cfg.n_kv_heads, cfg.head_dim)
    v = f(u @ w["wv"].T).reshape(T, cfg.n_kv_heads, cfg.head_dim)
    c, s = rope_angles(pos, cfg.head_dim, cfg.rope_base)
    q, k = f(apply_rope(q, c, s)), f(apply_rope(k, c, s))
    x = f(x + f(attention(q, k, v, pos, pos)) @ w["wo"].T)
    u = f(rms_norm(x, 1.0, cfg.rms_eps))
    x = f(x + f(silu(u @ w["wgate"].T) * (u @ w["wup"].T)) @ w["wdown"].T)
    err = np.linalg.norm(x - ref) / np.linalg.norm(ref)
    assert 1e-2 < err < 2e-2, err
