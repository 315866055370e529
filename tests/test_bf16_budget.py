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


# ------------------------------------------------ the bf16-storage evaluator

import json  # noqa: E402
import os  # noqa: E402

from oracle.bf16eval import Bf16Stage, hidden_err  # noqa: E402
from oracle.llama import SyntheticWeights  # noqa: E402
from workloads import WORKLOADS  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bf16_budget.json")


def _tiny():
    cfg = WORKLOADS["tiny-2x1"].cfg
    return cfg, SyntheticWeights(cfg), gen.tokens(cfg.vocab, 20, 9)


def test_bf16_evaluator_without_rounding_is_the_oracle_bitwise():
    cfg, W, toks = _tiny()
    a, b = Stage(cfg, W, 0, cfg.n_layers), Bf16Stage(cfg, W, 0, cfg.n_layers, rounding=False)
    assert np.array_equal(a.prefill([0], [20], toks), b.prefill([0], [20], toks))
    for t in (3, 17):
        assert np.array_equal(a.decode([0], np.array([t])), b.decode([0], np.array([t])))


def test_bf16_evaluator_stores_bf16_and_stays_close():
    """Every cached key/value and every stage output is a bf16 value; the
    evaluation differs from the oracle by rounding-sized amounts (relative
    Frobenius error of the hidden state between 2^-10 and 2^-5 after one
    layer)."""
    cfg, W, toks = _tiny()
    st = Bf16Stage(cfg, W, 0, 1)
    h = st.prefill([0], [20], toks)
    for arr in (h, *st.kv[0][0]):
        assert np.array_equal(arr, gen.round_to_bf16(np.asarray(arr, np.float32)))
    err = hidden_err(h, Stage(cfg, W, 0, 1).prefill([0], [20], toks))
    assert 2.0 ** -10 < err < 2.0 ** -5, err


def test_budget_file_matches_the_evaluator():
    """tests/golden/bf16_budget.json is what tests/golden/make_bf16_budget.py
    writes: its first entry (7B shape, layers 0-7 from the embedding, 128
    tokens) is recomputed here for the first four layers. The errors grow
    with depth, and every entry the full-size GPU tests read is present."""
    import importlib.util
    with open(GOLDEN) as f:
        data = json.load(f)
    assert data["stated_logit_tol"] == 3e-2 and data["margin"] == 1.5
    ent = data["entries"]
    for name in ("7b_l0-8_t128", "c2_7b_l8-16_p512", "c3_7b_full_seq0_p1024",
                 "c4_13b_full_seq1_p2048", "c5_8b_full_shortest", "c5_8b_full_longest"):
        assert name in ent, name
    for name in ("7b_l0-8_t128", "c2_7b_l8-16_p512"):
        e = ent[name]["hidden_err_after_layer"]
        assert all(x < y for x, y in zip(e, e[1:])), name
    spec = importlib.util.spec_from_file_location(
        "make_bf16_budget", os.path.join(os.path.dirname(GOLDEN), "make_bf16_budget.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    got = mod.entry_7b_first_layers(n_layers=4)["hidden_err_after_layer"]
    want = ent["7b_l0-8_t128"]["hidden_err_after_layer"][:4]
    assert np.allclose(got, want, rtol=2e-2), (got, want)
