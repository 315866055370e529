"""Writes tests/golden/bf16_budget.json: how far a bfloat16-storage
evaluation of each full-size check drifts from the float32 oracle.

The full-size GPU tests compare the engine with the float32 oracle. The
engine stores weights and activations in bfloat16 (one 16-bit hidden vector
per token at the stage boundary, as section 4.1 prices it), so over 32-40
layers part of its difference from the oracle is the rounding of what it
stores, whatever the kernels do. This script evaluates exactly the sequences
those tests check with ``oracle.bf16eval.Bf16Stage`` (the oracle's steps,
with the stored tensors rounded) and with the float32 oracle, and records
the difference. The tests then allow max(stated tolerance, MARGIN x this
difference). Only ``oracle/`` and the seeded generators are used.

    python tests/golden/make_bf16_budget.py            # all entries (~15 min, ~40 GB)
    python tests/golden/make_bf16_budget.py 7b_l0-8_t128   # one entry
"""
from __future__ import annotations

import concurrent.futures as cf
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle.bf16eval import Bf16Stage, hidden_err, logit_err  # noqa: E402
from oracle.llama import Stage, argmax_lowest  # noqa: E402
from workloads import MODELS, WORKLOADS, gen  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "bf16_budget.json")
STATED = 3e-2   # logits max|err| <= 3e-2 * max|logit|
MARGIN = 1.5
KINDS = ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")


class LayerWeights:
    """float32 draws of the given layers (+ embedding / head), generated in
    parallel and kept."""

    def __init__(self, cfg, layers, embed, head, threads=8):
        self.cfg = cfg
        items = [(l, k) for l in layers for k in KINDS]
        if embed:
            items.append((-1, "embed"))
        if head:
            items.append((-1, "lm_head"))
        with cf.ThreadPoolExecutor(threads) as ex:
            arrs = list(ex.map(lambda it: gen.weight_f32(cfg, *it), items))
        self.w = dict(zip(items, arrs))

    def __call__(self, layer, kind):
        if kind in ("attn_norm", "ffn_norm", "final_norm"):
            return gen.gains(self.cfg)
        return self.w[(-1, kind) if kind in ("embed", "lm_head") else (layer, kind)]


def chain(cfg, begin, end, inp, embed_head_in_range=True, per_layer=False):
    """Float32 oracle and bf16 evaluation of layers [begin, end) on one
    sequence, one layer's weights in memory at a time (single-layer stages
    chained give the oracle's full-range result bit for bit). Returns the
    two outputs and, if asked, the hidden error after every layer."""
    xo, xe, errs = inp, inp, []
    for l in range(begin, end):
        W = LayerWeights(cfg, [l], embed=(l == 0), head=(l == cfg.n_layers - 1))
        n = len(inp)
        xo = Stage(cfg, W, l, l + 1).prefill([0], [n], xo)
        xe = Bf16Stage(cfg, W, l, l + 1).prefill([0], [n], xe)
        if per_layer and l < cfg.n_layers - 1:
            errs.append(hidden_err(xe, xo))
        del W
    return xo, xe, errs


def entry_7b_first_layers(n_layers=8, T=128):
    """Layers [0, n) of the 7B shape from the embedding, 128 tokens: the
    hidden error after every layer (recomputed by the CPU test)."""
    cfg = MODELS["llama2-7b"]
    toks = gen.tokens(cfg.vocab, T, 3)
    _, _, errs = chain(cfg, 0, n_layers, toks, per_layer=True)
    return {"model": "llama2-7b", "layers": [0, n_layers], "tokens": T, "token_seed": 3,
            "hidden_err_after_layer": errs}


def entry_c2(steps=2):
    """The 7B middle stage (layers 8-15) on a 512-token prompt: its input is
    the oracle's output of layers 0-7 on the prompt, rounded to bf16; the
    oracle and the bf16 evaluation both start from that input. Then two
    decode steps whose inputs are the oracle's layers 0-7 on tokens drawn
    from stream [1, 100 + step], rounded to bf16."""
    wl = WORKLOADS["7b-stage8-15-cold"]
    cfg = wl.cfg
    b, e = wl.stages[wl.bench_stage]
    P = wl.prompt_lens[0]
    toks = gen.tokens(cfg.vocab, P, wl.seed)
    W0 = LayerWeights(cfg, range(0, b), embed=True, head=False)
    first = Stage(cfg, W0, 0, b)
    x8 = gen.round_to_bf16(first.prefill([0], [P], toks).astype(np.float32))
    dec_in = []
    for s in range(steps):
        t = gen.tokens(cfg.vocab, 1, 100 + s)
        dec_in.append(gen.round_to_bf16(first.decode([0], t).astype(np.float32)))
    del W0, first
    W = LayerWeights(cfg, range(b, e), embed=False, head=False)
    errs = []
    xo, xe = x8, x8
    for l in range(b, e):   # per layer, single-layer stages
        xo = Stage(cfg, W, l, l + 1).prefill([0], [P], xo)
        xe = Bf16Stage(cfg, W, l, l + 1).prefill([0], [P], xe)
        errs.append(hidden_err(xe, xo))
    o, m = Stage(cfg, W, b, e), Bf16Stage(cfg, W, b, e)
    o.prefill([0], [P], x8)
    m.prefill([0], [P], x8)
    dec = [hidden_err(m.decode([0], d), o.decode([0], d)) for d in dec_in]
    return {"workload": wl.name, "layers": [b, e], "tokens": P,
            "input": "bf16(oracle layers 0-7 on the prompt)", "hidden_err_after_layer": errs,
            "decode_hidden_err": dec,
            "decode_input": "bf16(oracle layers 0-7 decoding token gen.tokens(V, 1, 100 + step))"}


def whole_model(cfg, toks, decode_steps):
    """Prefill of one sequence through the whole model, then greedy decode
    steps fed with the oracle's tokens (teacher forcing of the bf16
    evaluation). Returns the logit errors of the prefill's last position and
    of each step, and the oracle's tokens and top-2 margins."""
    W = LayerWeights(cfg, range(cfg.n_layers), embed=True, head=True)
    o = Stage(cfg, W, 0, cfg.n_layers)
    e = Bf16Stage(cfg, W, 0, cfg.n_layers)
    lo = o.prefill([0], [len(toks)], toks)[-1]
    le = e.prefill([0], [len(toks)], toks)[-1]
    errs, toks_o, margins = [logit_err(le, lo)], [], []
    for s in range(decode_steps + 1):
        t = int(argmax_lowest(lo))
        top2 = np.sort(lo)[-2:]
        toks_o.append(t)
        margins.append(float((top2[1] - top2[0]) / np.abs(lo).max()))
        if s == decode_steps:
            break
        lo = o.decode([0], np.array([t], np.int32))[0]
        le = e.decode([0], np.array([t], np.int32))[0]
        errs.append(logit_err(le, lo))
    del W
    return errs, toks_o, margins


def entry_c3(steps=3):
    """7B, all 32 layers + head: sequence 0 of the batch-8 x 1024 prompt."""
    wl = WORKLOADS["7b-full-b8"]
    cfg = wl.cfg
    P = wl.prompt_lens[0]
    toks = gen.tokens(cfg.vocab, wl.batch * P, wl.seed)[:P]
    errs, t, m = whole_model(cfg, toks, steps)
    return {"workload": wl.name, "sequence": 0, "tokens": P, "logit_err": errs,
            "oracle_tokens": t, "oracle_top2_margin": m}


def entry_c4():
    """13B, both 20-layer stages: sequence 1 of the batch-4 x 2048 prompt
    (prefill only; one layer in memory at a time)."""
    wl = WORKLOADS["13b-2x20-b4"]
    cfg = wl.cfg
    P = wl.prompt_lens[0]
    toks = gen.tokens(cfg.vocab, wl.batch * P, wl.seed)[P:2 * P]
    lo, le, _ = chain(cfg, 0, cfg.n_layers, toks)
    return {"workload": wl.name, "sequence": 1, "tokens": P,
            "logit_err": [logit_err(le[-1], lo[-1])]}


def entry_c5(which, steps):
    """8B-GQA, all 32 layers + head: the shortest or longest ragged prompt."""
    wl = WORKLOADS["8b-4x8-ragged-merge"]
    cfg = wl.cfg
    lens = wl.lengths()
    i = int(np.argmin(lens)) if which == "shortest" else int(np.argmax(lens))
    starts = np.concatenate([[0], np.cumsum(lens)])
    toks = gen.tokens(cfg.vocab, sum(lens), wl.seed)[starts[i]:starts[i + 1]]
    errs, t, m = whole_model(cfg, toks, steps)
    return {"workload": wl.name, "sequence": i, "tokens": int(lens[i]), "logit_err": errs,
            "oracle_tokens": t, "oracle_top2_margin": m}


ENTRIES = {
    "7b_l0-8_t128": entry_7b_first_layers,
    "c2_7b_l8-16_p512": entry_c2,
    "c3_7b_full_seq0_p1024": entry_c3,
    "c5_8b_full_shortest": lambda: entry_c5("shortest", 3),
    "c5_8b_full_longest": lambda: entry_c5("longest", 0),
    "c4_13b_full_seq1_p2048": entry_c4,
}


def main(names):
    data = {"stated_logit_tol": STATED, "margin": MARGIN, "entries": {}}
    if os.path.exists(OUT):
        with open(OUT) as f:
            data["entries"] = json.load(f).get("entries", {})
    for name in names:
        t = time.time()
        data["entries"][name] = ENTRIES[name]()
        print(f"{name}: {data['entries'][name]} ({time.time() - t:.0f} s)", flush=True)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1)


if __name__ == "__main__":
    main(sys.argv[1:] or list(ENTRIES))
