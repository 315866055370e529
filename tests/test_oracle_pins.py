"""Pins for the CPU oracle: brute force, invariants, closed forms, library
cross-checks and sizes printed in the paper. These run without a GPU.
"""
import dataclasses
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import kvblob
from oracle.llama import (Stage, SyntheticWeights, apply_rope, attention,
                          attention_probs, full_forward, greedy_generate,
                          rms_norm, rope_angles, argmax_lowest)
from workloads import MODELS, ModelCfg, gen
from tests.bruteforce import BruteDecoder

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# Tiny shapes for brute force: GQA (4 query heads over 2 KV heads) and MHA.
PIN_GQA = ModelCfg("pin-gqa", n_layers=2, hidden=16, n_heads=4, n_kv_heads=2,
                   head_dim=4, ffn=24, vocab=32)
PIN_MHA = ModelCfg("pin-mha", n_layers=2, hidden=16, n_heads=2, n_kv_heads=2,
                   head_dim=8, ffn=24, vocab=32, rope_base=100.0)


class Scaled(SyntheticWeights):
    """Larger weight scale so that tiny models have non-trivial attention."""

    def __call__(self, layer, kind):
        w = super().__call__(layer, kind)
        if kind.startswith("w") or kind in ("embed", "lm_head"):
            return w * np.float32(25.0)
        return w


# ------------------------------------------------------------ P1 brute force

@pytest.mark.parametrize("cfg", [PIN_GQA, PIN_MHA], ids=lambda c: c.name)
def test_bruteforce_full_forward(cfg):
    W = Scaled(cfg)
    toks = gen.tokens(cfg.vocab, 6, 11)
    ref = np.array(BruteDecoder(cfg, W).logits(list(toks)))
    o64 = full_forward(cfg, W, toks, dtype=np.float64)
    o32 = full_forward(cfg, W, toks, dtype=np.float32)
    scale = np.max(np.abs(ref))
    assert np.max(np.abs(o64 - ref)) <= 1e-12 * scale
    assert np.max(np.abs(o32 - ref)) <= 1e-5 * scale


def test_bruteforce_middle_stage_hidden():
    cfg = dataclasses.replace(PIN_GQA, n_layers=3)
    W = Scaled(cfg)
    x = gen.hidden_input(5, cfg.hidden, 3).astype(np.float64)
    ref = np.array(BruteDecoder(cfg, W).hidden_after(1, 2, x.tolist()))
    st = Stage(cfg, W, 1, 2, dtype=np.float64)
    out = st.prefill([7], [5], x)
    assert np.max(np.abs(out - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_bruteforce_decode_with_cache():
    cfg = PIN_GQA
    W = Scaled(cfg)
    toks = list(gen.tokens(cfg.vocab, 7, 12))
    ref = np.array(BruteDecoder(cfg, W).logits(toks))
    st = Stage(cfg, W, 0, cfg.n_layers, dtype=np.float64)
    st.prefill([1], [4], np.array(toks[:4]))
    for t in range(4, 7):
        lg = st.decode([1], np.array([toks[t]]))
        assert np.max(np.abs(lg[0] - ref[t])) <= 1e-12 * np.max(np.abs(ref))


# --------------------------------------------------------------- invariants

def test_split_equals_full_bitwise():
    cfg = MODELS["tiny"]
    W = SyntheticWeights(cfg)
    toks = gen.tokens(cfg.vocab, 20, 5)
    full = Stage(cfg, W, 0, 2).prefill([0], [20], toks)
    a = Stage(cfg, W, 0, 1).prefill([0], [20], toks)
    b = Stage(cfg, W, 1, 2).prefill([0], [20], a)
    assert np.array_equal(full, b)


@pytest.mark.parametrize("dtype,tol", [(np.float64, 1e-12), (np.float32, 1e-5)])
def test_prefill_then_decode_equals_recompute(dtype, tol):
    cfg = MODELS["tiny"]
    W = SyntheticWeights(cfg)
    prompt = gen.tokens(cfg.vocab, 12, 6)
    toks, logits = greedy_generate(cfg, W, prompt, 5, stages=[(0, 1), (1, 2)],
                                   dtype=dtype)
    seq = np.concatenate([prompt, toks[:-1]])
    ref = full_forward(cfg, W, seq, dtype=dtype)[len(prompt) - 1:]
    assert np.max(np.abs(logits - ref)) <= tol * np.max(np.abs(ref))


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((9, 16)).astype(np.float32)
    k = rng.standard_normal((9, 16)).astype(np.float32) * 4
    p = attention_probs(q, k, np.arange(9), np.arange(9), 0.25)
    assert np.max(np.abs(p.sum(axis=1) - 1)) <= 1e-6
    assert np.all(np.triu(p, 1) == 0)


def test_causality_bitwise():
    cfg = MODELS["tiny"]
    W = SyntheticWeights(cfg)
    toks = gen.tokens(cfg.vocab, 24, 7)
    base = full_forward(cfg, W, toks)
    j = 15
    t2 = toks.copy()
    t2[j] = (t2[j] + 1) % cfg.vocab
    pert = full_forward(cfg, W, t2)
    assert np.array_equal(base[:j], pert[:j])
    assert not np.array_equal(base[j], pert[j])


# ------------------------------------------------------------- closed forms

def test_zero_attention_and_mlp_gives_embedding_logits():
    cfg = PIN_GQA
    base = SyntheticWeights(cfg)

    def W(layer, kind):
        w = base(layer, kind)
        return np.zeros_like(w) if kind in ("wo", "wdown") else w

    toks = gen.tokens(cfg.vocab, 5, 8)
    out = full_forward(cfg, W, toks, dtype=np.float64)
    E = base(-1, "embed").astype(np.float64)[toks]
    rms = np.sqrt((E ** 2).mean(axis=1, keepdims=True) + cfg.rms_eps)
    ref = (E / rms) @ base(-1, "lm_head").astype(np.float64).T
    assert np.allclose(out, ref, rtol=0, atol=1e-12 * np.abs(ref).max())


def test_one_token_attention_returns_v():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 4, 8))
    k = rng.standard_normal((1, 2, 8))
    v = rng.standard_normal((1, 2, 8))
    o = attention(q, k, v, np.array([0]), np.array([0])).reshape(1, 4, 8)
    for h in range(4):
        assert np.array_equal(o[0, h], v[0, h // 2])


def test_identical_keys_average_values():
    rng = np.random.default_rng(2)
    n = 6
    q = rng.standard_normal((n, 1, 8))
    k = np.repeat(rng.standard_normal((1, 1, 8)), n, axis=0)
    v = rng.standard_normal((n, 1, 8))
    o = attention(q, k, v, np.arange(n), np.arange(n))
    for i in range(n):
        assert np.allclose(o[i], v[:i + 1, 0].mean(axis=0), atol=1e-14)


def test_rope_closed_forms():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 3, 16))
    cos, sin = rope_angles(np.zeros(5), 16, 10000.0)
    assert np.array_equal(apply_rope(x, cos, sin), x)       # position 0
    pos = np.array([0, 1, 5, 17, 300])
    cos, sin = rope_angles(pos, 16, 10000.0)
    y = apply_rope(x, cos, sin)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1))
    # d = 2: a plain rotation of (x0, x1) by pos radians (theta_0 = 1)
    v = np.array([[[0.3, -1.2]]])
    c, s = rope_angles([2.0], 2, 10000.0)
    r = apply_rope(v, c, s)[0, 0]
    assert np.allclose(r, [0.3 * math.cos(2) + 1.2 * math.sin(2),
                           -1.2 * math.cos(2) + 0.3 * math.sin(2)], atol=1e-15)
    # q_m . k_n depends only on m - n
    q = rng.standard_normal((1, 1, 16))
    k = rng.standard_normal((1, 1, 16))

    def dot(m, n):
        cm, sm = rope_angles([m], 16, 10000.0)
        cn, sn = rope_angles([n], 16, 10000.0)
        return float(np.sum(apply_rope(q, cm, sm) * apply_rope(k, cn, sn)))

    assert abs(dot(7, 3) - dot(104, 100)) < 1e-12
    assert abs(dot(7, 3) - dot(7, 2)) > 1e-6


def test_rmsnorm_unit_rms():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((7, 64)) * 3
    y = rms_norm(x, np.ones(64), 1e-5)
    ms = (x ** 2).mean(axis=1)
    assert np.allclose(np.sqrt((y ** 2).mean(axis=1)), np.sqrt(ms / (ms + 1e-5)),
                       atol=1e-14)


def test_argmax_lowest_index_on_ties():
    assert argmax_lowest(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    assert list(argmax_lowest(np.array([[0.0, 0.0], [1.0, 2.0]]))) == [0, 1]


# -------------------------------------------------- P4 library cross-checks

def test_attention_matches_torch_sdpa_and_rms_norm():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    T, nh, nkv, d = 11, 4, 2, 16
    q = rng.standard_normal((T, nh, d))
    k = rng.standard_normal((T, nkv, d))
    v = rng.standard_normal((T, nkv, d))
    o = attention(q, k, v, np.arange(T), np.arange(T)).reshape(T, nh, d)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(np.repeat(k, 2, axis=1)).permute(1, 0, 2)
    tv = torch.from_numpy(np.repeat(v, 2, axis=1)).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, is_causal=True).permute(1, 0, 2).numpy()
    assert np.max(np.abs(o - ref)) < 1e-12
    x = rng.standard_normal((5, 32))
    g = rng.standard_normal(32)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (32,),
                                       torch.from_numpy(g), eps=1e-5).numpy()
    assert np.max(np.abs(rms_norm(x, g, 1e-5) - ref)) < 1e-12


# ---------------------------------------------------- P5 paper-printed sizes

def test_paper_printed_model_sizes():
    with open(os.path.join(GOLDEN, "paper_sizes.json")) as f:
        g = json.load(f)
    for name, exact in (("llama2-7b", 13_476_831_232),
                        ("llama2-13b", 26_031_728_640)):
        b = oracle.image_bytes_16bit(MODELS[name])
        assert b == exact
        printed = g[name]["model_size_printed_gib"]
        assert math.floor(b / 2 ** 30 * 10) / 10 == printed
    assert oracle.boundary_bytes_per_token(MODELS["llama2-7b"]) == \
        g["llama2-7b-boundary"]["bytes_per_token_printed_kib"] * 1024


def test_stage_partition_covers_model_exactly():
    cfg = MODELS["llama2-7b"]
    parts = sum(oracle.param_count(cfg, b, e) for b, e in
                ((0, 8), (8, 16), (16, 24), (24, 32)))
    assert parts == oracle.param_count(cfg)
    assert oracle.image_bytes_16bit(cfg, 8, 16) == 3_238_133_760


# ---------------------------------------------------------- KV blob codec

def test_kvblob_field_offsets_and_roundtrip():
    rng = np.random.default_rng(6)
    seqs = []
    for sid, n in ((42, 5), (-3, 16), (7, 17)):
        k = rng.integers(0, 65536, (2, n, 3, 8), dtype=np.uint16)
        v = rng.integers(0, 65536, (2, n, 3, 8), dtype=np.uint16)
        seqs.append((sid, k, v))
    blob = kvblob.pack(4, 6, 3, 8, 16, seqs)
    assert blob[:4] == b"HSKV"
    assert int.from_bytes(blob[12:16], "little", signed=True) == 4
    assert int.from_bytes(blob[16:20], "little", signed=True) == 6
    assert int.from_bytes(blob[32:36], "little") == 3
    poff = int.from_bytes(blob[40:48], "little")
    assert poff == 256 and len(blob) == int.from_bytes(blob[56:64], "little")
    assert int.from_bytes(blob[64:72], "little", signed=True) == 42
    assert int.from_bytes(blob[72:76], "little") == 5
    assert int.from_bytes(blob[76:80], "little") == 1
    # blocks: 1 + 1 + 2 per layer, K and V, each [3][16][8] bf16
    assert len(blob) - poff == 2 * 4 * 2 * 3 * 16 * 8 * 2
    assert len(blob) == kvblob.blob_size(2, 3, 8, 16, [5, 16, 17])
    # first K block of seq 42, head 1, slot 2 = K[layer 0][token 2][head 1]
    first = np.frombuffer(blob, np.uint16, offset=poff, count=3 * 16 * 8)
    first = first.reshape(3, 16, 8)
    assert np.array_equal(first[1, 2], seqs[0][1][0, 2, 1])
    assert np.all(first[:, 5:, :] == 0)                      # padded slots
    hdr, out = kvblob.parse(blob)
    assert hdr["records"] == [(42, 5, 1), (-3, 16, 1), (7, 17, 2)]
    for (sid, k, v), (sid2, k2, v2) in zip(seqs, out):
        assert sid == sid2 and np.array_equal(k, k2) and np.array_equal(v, v2)
    with pytest.raises(ValueError):
        kvblob.parse(blob[:-2])


def test_ragged_workload_block_count():
    lens = gen.ragged_lengths(128, 2048, 16, 0)
    assert sum(lens) == 17543
    assert sum(-(-n // 16) for n in lens) == 1102


# ----------------------------------------------------- input generators

def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 1 + 2 ** -7 + 2 ** -9],
                 dtype=np.float32)
    r = gen.round_to_bf16(x)
    assert list(r) == [1.0, 1.0, 1 + 2 ** -6, -2.5, 1 + 2 ** -7]


def test_generators_are_seeded_and_per_tensor():
    cfg = MODELS["tiny"]
    a = gen.weight_f32(cfg, 1, "wq")
    assert np.array_equal(a, gen.weight_f32(cfg, 1, "wq"))
    assert not np.array_equal(a, gen.weight_f32(cfg, 0, "wq"))
    assert a.shape == (256, 256) and a.dtype == np.float32
    assert abs(float(a.std()) - 0.02) < 0.001
    t = gen.tokens(1024, 32, 1)
    assert t.min() >= 0 and t.max() < 1024 and np.array_equal(t, gen.tokens(1024, 32, 1))
