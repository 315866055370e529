"""Parity at the full workload sizes, in the launch configurations the
benchmark and the serving path use.

Two kinds of checks against the float32 oracle:

* One layer at a time, on the engine's own inputs to that layer: a layer
  range cut into single-layer stages gives, bitwise, the same results as the
  uncut range (checked here too), so those stages expose the inputs and
  outputs of individual layers of the launch configuration. Per layer the
  hidden state is within HIDDEN_TOL and the last layer + head within the
  stated logit tolerance.
* End to end, whole stacks from the tokens (teacher-forced on the engine's
  tokens in decode). Over 8-40 layers a bf16-storage evaluation itself
  drifts from the float32 definition; tests/golden/bf16_budget.json holds,
  for exactly these sequences, how far the CPU's bf16-storage evaluation of
  the oracle (oracle/bf16eval.py) is from the float32 oracle. The bound is
  max(stated tolerance, MARGIN x that), so the stated 3e-2 applies wherever
  bf16 storage can meet it.

Properties that hold at any size (split == full, merged == pipeline, export
-> import -> export, cold == warm) are checked bitwise on everything.
"""
import concurrent.futures as cf
import gc
import json
import os
import time

import numpy as np
import pytest

from oracle import kvblob
from oracle.llama import Stage as OStage
from workloads import WORKLOADS, gen
from tests import gpu_util as G

pytestmark = [pytest.mark.gpu, pytest.mark.big]
LOGIT_TOL = 3e-2           # max|err| / max|logit| (the stated tolerance)
# One layer, relative Frobenius error of its output hidden state: a
# bf16-storage evaluation of a single layer of these shapes is off by up to
# 1.2% (layer 0 fed from the embedding, whose output is all new content), so
# the bound is 2e-2; deeper layers measure 0.3-0.6%.
HIDDEN_TOL = 2e-2
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                       "bf16_budget.json")) as _f:
    BUDGET = json.load(_f)


def logit_bound(entry, i):
    """Logit tolerance for check i of a budget entry (prefill = 0, then the
    decode steps)."""
    e = BUDGET["entries"][entry]["logit_err"]
    return max(BUDGET["stated_logit_tol"], BUDGET["margin"] * e[min(i, len(e) - 1)])


def hidden_bound(vals):
    return max(1e-2, BUDGET["margin"] * max(vals))


T0 = time.time()


def say(*a):
    print(f"[{time.time() - T0:7.1f}s]", *a, flush=True)


class Weights:
    """float32 draws of ``workloads.gen`` for the given layers (+ embedding /
    head), generated in parallel and shared by the oracle and the packer."""

    def __init__(self, cfg, layers, embed=False, head=False, threads=16):
        self.cfg = cfg
        items = [(l, k) for l in layers
                 for k in ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")]
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
        key = (-1, kind) if kind in ("embed", "lm_head") else (layer, kind)
        return self.w[key]


class Pipeline:
    """Stages for the given layer cuts, loaded from pinned images."""

    def __init__(self, cfg, cuts, W, **kw):
        from paper_2502_15524_amd import pipeline
        self.cfg, self.stages = cfg, []
        for b, e in cuts:
            st = pipeline.Stage(cfg, b, e, **kw)
            img = pipeline.pinned_image(cfg, b, e, source=W)
            st.load(img, 64 << 20)
            st.sync()
            img.close()
            self.stages.append(st)

    def prefill(self, ids, lens, inp):
        """Returns the host outputs of every stage (hidden [T, H] float32, or
        logits [n, V] for the last stage) and the next tokens (device)."""
        torch = G.torch()
        cfg, sp = self.cfg, G.stream_ptr()
        T, B = sum(lens), len(ids)
        x, outs = inp, []
        nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
        for st in self.stages:
            if st.end == cfg.n_layers:
                lg = torch.zeros((B, cfg.vocab), dtype=torch.float32, device="cuda")
                st.prefill(ids, lens, x.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
                outs.append(lg.cpu().numpy())
            else:
                out = torch.zeros((T, cfg.hidden), dtype=torch.bfloat16, device="cuda")
                st.prefill(ids, lens, x.data_ptr(), out.data_ptr(), 0, sp)
                outs.append(G.from_dev_bf16(out))
                x = out
        torch.cuda.synchronize()
        return outs, nxt

    def decode(self, ids, nxt):
        torch = G.torch()
        cfg, sp, B = self.cfg, G.stream_ptr(), len(ids)
        x, outs = nxt.clone(), []
        for st in self.stages:
            if st.end == cfg.n_layers:
                lg = torch.zeros((B, cfg.vocab), dtype=torch.float32, device="cuda")
                st.decode(ids, x.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
                outs.append(lg.cpu().numpy())
            else:
                out = torch.zeros((B, cfg.hidden), dtype=torch.bfloat16, device="cuda")
                st.decode(ids, x.data_ptr(), out.data_ptr(), 0, sp)
                outs.append(G.from_dev_bf16(out))
                x = out
        torch.cuda.synchronize()
        return outs

    def close(self):
        for st in self.stages:
            st.close()
        self.stages = []


def check_layer(cfg, W, layer, x_in, gpu_out, n_tok, head=False, tag=""):
    """Oracle layer `layer` (and the head) on the engine's input rows."""
    first = layer == 0
    ost = OStage(cfg, W, layer, layer + 1)
    ref = ost.prefill([0], [n_tok], x_in)
    if head:
        err = np.abs(gpu_out - ref[-1]).max() / np.abs(ref[-1]).max()
        say(f"{tag} layer {layer} + head: rel logit err {err:.2e}")
        assert err <= LOGIT_TOL
    else:
        err = G.rel_fro(gpu_out, ref)
        say(f"{tag} layer {layer}{' (from tokens)' if first else ''}: hidden err {err:.2e}")
        assert err <= HIDDEN_TOL
    return ost


def test_7b_middle_stage_512_per_layer_and_cold_equals_warm():
    """Layers 8-15 of the 7B shape, one 512-token prompt (the benchmark's
    workload), fed the oracle's output of layers 0-7 on the prompt (bf16):
    cold streaming == warm == in place (input and output in one buffer),
    8 single-layer stages == the stage, every layer
    against the oracle, KV through the export blob, the whole stage and two
    decode steps against the oracle end to end."""
    torch = G.torch()
    from paper_2502_15524_amd import hs, pipeline
    wl = WORKLOADS["7b-stage8-15-cold"]
    cfg = wl.cfg
    b, e = wl.stages[wl.bench_stage]
    P = wl.prompt_lens[0]
    say("oracle layers 0-7 on the prompt")
    W0 = Weights(cfg, range(0, b), embed=True)
    first = OStage(cfg, W0, 0, b)
    x32 = gen.round_to_bf16(first.prefill([0], [P], gen.tokens(cfg.vocab, P, wl.seed)))
    dec_in = [gen.round_to_bf16(first.decode([0], gen.tokens(cfg.vocab, 1, 100 + s)))
              for s in range(2)]
    del W0, first
    gc.collect()
    say("generating weights")
    W = Weights(cfg, range(b, e))
    kw = dict(max_seqs=4, max_ctx=P + 8, max_batch_tokens=P)
    st = pipeline.Stage(cfg, b, e, **kw)
    img = pipeline.pinned_image(cfg, b, e, source=W)
    x = G.to_dev_bf16(x32)
    sp = G.stream_ptr()
    outs = []
    for i in range(2):                       # cold: prefill enqueued while chunks fly
        hs.hs_stage_invalidate_weights(st.h)
        st.load(img, 64 << 20)
        out = torch.zeros((P, cfg.hidden), dtype=torch.bfloat16, device="cuda")
        st.prefill([i], [P], x.data_ptr(), out.data_ptr(), 0, sp)
        torch.cuda.synchronize()
        outs.append(G.from_dev_bf16(out))
    out = torch.zeros((P, cfg.hidden), dtype=torch.bfloat16, device="cuda")
    st.prefill([2], [P], x.data_ptr(), out.data_ptr(), 0, sp)      # warm
    torch.cuda.synchronize()
    warm = G.from_dev_bf16(out)
    assert np.array_equal(outs[0], warm) and np.array_equal(outs[1], warm)
    inout = x.clone()                        # input and output in one buffer
    st.prefill([3], [P], inout.data_ptr(), inout.data_ptr(), 0, sp)
    torch.cuda.synchronize()
    assert np.array_equal(G.from_dev_bf16(inout), warm)
    n = hs.hs_kv_export_size(st.h, [2])
    blob = torch.zeros(n, dtype=torch.uint8, device="cuda")
    hs.hs_kv_export(st.h, [2], blob.data_ptr(), n, sp)
    torch.cuda.synchronize()
    _, kv = kvblob.parse(blob.cpu().numpy().tobytes())
    dec_out = []
    for s in range(2):
        od = torch.zeros((1, cfg.hidden), dtype=torch.bfloat16, device="cuda")
        st.decode([2], G.to_dev_bf16(dec_in[s]).data_ptr(), od.data_ptr(), 0, sp)
        io = G.to_dev_bf16(dec_in[s])        # the same step in place, on the twin sequence
        st.decode([3], io.data_ptr(), io.data_ptr(), 0, sp)
        torch.cuda.synchronize()
        dec_out.append(G.from_dev_bf16(od))
        assert np.array_equal(G.from_dev_bf16(io), dec_out[-1])
    st.close()
    img.close()
    say("single-layer stages")
    pipe = Pipeline(cfg, [(l, l + 1) for l in range(b, e)], W, **kw)
    layer_out, _ = pipe.prefill([2], [P], x)
    assert np.array_equal(layer_out[-1], warm)              # split == full, bitwise
    pipe.close()
    say("oracle, layer by layer")
    inputs = [x32] + layer_out[:-1]
    osts = [check_layer(cfg, W, l, inputs[l - b], layer_out[l - b], P) for l in range(b, e)]
    # KV of each layer as exported, against the oracle on the same inputs
    for li in (0, e - b - 1):
        K, V = osts[li].kv[0][b + li]
        kg, vg = gen.bf16_bits_to_f32(kv[0][1][li]), gen.bf16_bits_to_f32(kv[0][2][li])
        assert np.abs(kg - K).max() <= 2e-2 * np.abs(K).max()
        assert np.abs(vg - V).max() <= 2e-2 * np.abs(V).max()
    # the whole stage against the oracle from the same input
    ent = BUDGET["entries"]["c2_7b_l8-16_p512"]
    ref = OStage(cfg, W, b, e)
    full = ref.prefill([0], [P], x32)
    drift = G.rel_fro(warm, full)
    bound = hidden_bound(ent["hidden_err_after_layer"][-1:])
    say(f"8-layer stage vs oracle {drift:.2e} (bf16 evaluation "
        f"{ent['hidden_err_after_layer'][-1]:.2e}, bound {bound:.2e})")
    assert drift <= bound
    dbound = hidden_bound(ent["decode_hidden_err"] + ent["hidden_err_after_layer"][-1:])
    for s in range(2):
        d = G.rel_fro(dec_out[s], ref.decode([0], dec_in[s]))
        say(f"decode step {s} vs oracle {d:.2e} (bound {dbound:.2e})")
        assert d <= dbound
    del W
    gc.collect()


def test_7b_full_batch8_prompt1024_decode():
    """All 32 layers + head of the 7B shape, batch 8 x 1024 prompt tokens,
    then 3 greedy decode steps over the paged cache. The model cut at layers
    1, 16, 17 and 31 gives the same logits bitwise; layers 0, 16 and 31 +
    head are checked against the oracle on sequence 0, for the prefill and
    for every decode step."""
    torch = G.torch()
    wl = WORKLOADS["7b-full-b8"]
    cfg = wl.cfg
    B, P, L = wl.batch, wl.prompt_lens[0], cfg.n_layers
    say("generating weights")
    W = Weights(cfg, range(L), embed=True, head=True)
    kw = dict(max_seqs=B, max_ctx=P + 16, max_batch_tokens=B * P)
    toks = gen.tokens(cfg.vocab, B * P, wl.seed)
    ids = list(range(B))
    x = torch.from_numpy(toks).cuda()
    full = Pipeline(cfg, [(0, L)], W, **kw)
    (f_logits,), nxt = full.prefill(ids, [P] * B, x)
    f_dec = []
    for _ in range(3):
        f_dec.append(full.decode(ids, nxt)[0])
    gtok = [int(np.argmax(f_logits[0]))] + [int(np.argmax(d[0])) for d in f_dec]
    full.close()
    say("cut pipeline")
    cuts = [(0, 1), (1, 16), (16, 17), (17, 31), (31, 32)]
    pipe = Pipeline(cfg, cuts, W, **kw)
    p_out, nxt = pipe.prefill(ids, [P] * B, x)
    assert np.array_equal(p_out[-1], f_logits)
    p_dec = []
    for s in range(3):
        p_dec.append(pipe.decode(ids, nxt))
        assert np.array_equal(p_dec[-1][-1], f_dec[s])
    pipe.close()
    gc.collect()
    say("oracle on sequence 0")
    rows = slice(0, P)
    o0 = check_layer(cfg, W, 0, toks[:P], p_out[0][rows], P, tag="prefill")
    o16 = check_layer(cfg, W, 16, p_out[1][rows], p_out[2][rows], P, tag="prefill")
    o31 = OStage(cfg, W, 31, 32)
    ref = o31.prefill([0], [P], p_out[3][rows])[-1]
    err = np.abs(p_out[4][0] - ref).max() / np.abs(ref).max()
    say(f"prefill layer 31 + head: rel logit err {err:.2e}")
    assert err <= LOGIT_TOL
    for s in range(3):
        d = p_dec[s]
        r0 = o0.decode([0], np.array([gtok[s]]))
        assert G.rel_fro(d[0][:1], r0) <= HIDDEN_TOL
        r16 = o16.decode([0], d[1][:1])
        assert G.rel_fro(d[2][:1], r16) <= HIDDEN_TOL
        r31 = o31.decode([0], d[3][:1])[0]
        err = np.abs(d[4][0] - r31).max() / np.abs(r31).max()
        say(f"decode step {s}: layer 31 + head rel logit err {err:.2e}")
        assert err <= LOGIT_TOL
    say("oracle end to end on sequence 0 (teacher-forced on the engine's tokens)")
    ent = "c3_7b_full_seq0_p1024"
    say(f"engine tokens {gtok}, oracle's greedy tokens in the budget run "
        f"{BUDGET['entries'][ent]['oracle_tokens']}")
    ow = OStage(cfg, W, 0, L)
    ref = ow.prefill([0], [P], toks[:P])[-1]
    got = [f_logits[0]] + [f_dec[s][0] for s in range(3)]
    refs = [ref] + [ow.decode([0], np.array([gtok[s]], np.int32))[0] for s in range(3)]
    for s, (g_, r_) in enumerate(zip(got, refs)):
        err = np.abs(g_ - r_).max() / np.abs(r_).max()
        say(f"32 layers + head, {'prefill' if s == 0 else f'decode step {s - 1}'}: "
            f"rel logit err {err:.2e} (bound {logit_bound(ent, s):.2e})")
        assert err <= logit_bound(ent, s)
    del W
    gc.collect()


def test_13b_two_stages_batch4_prompt2048():
    """13B shape as 2 stages of 20 layers, batch 4 x 2048. Cutting each stage
    once more (layers 0, 20 and 39 on their own) gives the same logits
    bitwise; those layers are checked against the oracle on sequence 1 over
    all 2048 positions."""
    torch = G.torch()
    wl = WORKLOADS["13b-2x20-b4"]
    cfg = wl.cfg
    B, P = wl.batch, wl.prompt_lens[0]
    say("generating weights")
    W = Weights(cfg, range(cfg.n_layers), embed=True, head=True)
    kw = dict(max_seqs=B, max_ctx=P + 8, max_batch_tokens=B * P)
    toks = gen.tokens(cfg.vocab, B * P, wl.seed)
    ids = list(range(B))
    x = torch.from_numpy(toks).cuda()
    two = Pipeline(cfg, list(wl.stages), W, **kw)
    (h20, logits2), _ = two.prefill(ids, [P] * B, x)
    two.close()
    gc.collect()
    say("cut pipeline")
    cuts = [(0, 1), (1, 20), (20, 21), (21, 39), (39, 40)]
    pipe = Pipeline(cfg, cuts, W, **kw)
    out, _ = pipe.prefill(ids, [P] * B, x)
    pipe.close()
    gc.collect()
    assert np.array_equal(out[1], h20) and np.array_equal(out[-1], logits2)
    say("oracle on sequence 1")
    i = 1
    rows = slice(i * P, (i + 1) * P)
    check_layer(cfg, W, 0, toks[rows], out[0][rows], P, tag="seq 1")
    check_layer(cfg, W, 20, out[1][rows], out[2][rows], P, tag="seq 1")
    ref = OStage(cfg, W, 39, 40).prefill([0], [P], out[3][rows])[-1]
    err = np.abs(out[4][i] - ref).max() / np.abs(ref).max()
    say(f"seq 1 layer 39 + head: rel logit err {err:.2e}")
    assert err <= LOGIT_TOL
    say("oracle end to end on sequence 1 (40 layers + head)")
    ref = OStage(cfg, W, 0, cfg.n_layers).prefill([0], [P], toks[rows])[-1]
    err = np.abs(logits2[i] - ref).max() / np.abs(ref).max()
    bound = logit_bound("c4_13b_full_seq1_p2048", 0)
    say(f"seq 1, both stages: rel logit err {err:.2e} (bound {bound:.2e})")
    assert err <= bound
    del W
    gc.collect()


def test_8b_gqa_four_stages_ragged_merge():
    """Llama-3-8B shape (GQA 32/8), 4 stages of 8 layers, 16 ragged prompts
    (sum 17,543 tokens): KV export -> import -> export is byte-identical for
    every stage, the merged worker decodes exactly like the pipeline, the
    last stage cut at layer 31 gives the same logits, and layer 31 + head is
    checked against the oracle on the shortest and the longest sequence."""
    torch = G.torch()
    from paper_2502_15524_amd import hs, pipeline
    wl = WORKLOADS["8b-4x8-ragged-merge"]
    cfg = wl.cfg
    lens = wl.lengths()
    B, T, L = len(lens), sum(lens), cfg.n_layers
    ids = list(range(100, 100 + B))
    say("generating weights")
    W = Weights(cfg, range(L), embed=True, head=True)
    toks = gen.tokens(cfg.vocab, T, wl.seed)
    sp = G.stream_ptr()
    kw = dict(max_seqs=B, max_ctx=max(lens) + 16, max_batch_tokens=T)
    x = torch.from_numpy(toks).cuda()
    say("pipeline A")
    A = Pipeline(cfg, list(wl.stages), W, **kw)
    a_out, nxt_a = A.prefill(ids, lens, x)
    say("pipeline B")
    Bp = Pipeline(cfg, list(wl.stages), W, **kw)
    b_out, nxt_b = Bp.prefill(ids, lens, x)
    assert np.array_equal(a_out[-1], b_out[-1])
    for st in Bp.stages:
        n = hs.hs_kv_export_size(st.h, ids)
        b1 = torch.zeros(n, dtype=torch.uint8, device="cuda")
        hs.hs_kv_export(st.h, ids, b1.data_ptr(), n, sp)
        fresh = pipeline.Stage(cfg, st.begin, st.end, **kw)
        hs.hs_kv_import(fresh.h, b1.data_ptr(), n, sp)
        b2 = torch.zeros(n, dtype=torch.uint8, device="cuda")
        hs.hs_kv_export(fresh.h, ids, b2.data_ptr(), n, sp)
        torch.cuda.synchronize()
        assert torch.equal(b1, b2)
        fresh.close()
        del b1, b2
    say("merging pipeline B into one worker")
    merged = pipeline.Stage(cfg, 0, 0, resident=(0, L), **kw)
    img = pipeline.pinned_image(cfg, 0, L, source=W)
    merged.load(img, 64 << 20)
    merged.sync()
    img.close()
    hs.hs_stage_merge(merged.h, [s.h for s in Bp.stages], sp)
    assert merged.info()["layer_end"] == L and merged.info()["live_seqs"] == B
    mp = Pipeline.__new__(Pipeline)
    mp.cfg, mp.stages = cfg, [merged]
    fed, merged_logits = [], []
    for s in range(3):
        fed.append(nxt_b.cpu().numpy().copy())
        la = A.decode(ids, nxt_a)[-1]
        lm = mp.decode(ids, nxt_b)[-1]
        assert np.array_equal(la, lm) and torch.equal(nxt_a, nxt_b)
        merged_logits.append(lm)
    A.close(), Bp.close(), mp.close()
    gc.collect()
    say("last stage cut at layer 31")
    C = Pipeline(cfg, [(0, 8), (8, 16), (16, 24), (24, 31), (31, 32)], W, **kw)
    c_out, _ = C.prefill(ids, lens, x)
    C.close()
    assert np.array_equal(c_out[-1], a_out[-1])
    starts = np.concatenate([[0], np.cumsum(lens)])
    o31 = OStage(cfg, W, 31, 32)
    for i in (int(np.argmin(lens)), int(np.argmax(lens))):
        rows = slice(starts[i], starts[i + 1])
        ref = o31.prefill([i], [lens[i]], c_out[3][rows])[-1]
        err = np.abs(c_out[4][i] - ref).max() / np.abs(ref).max()
        say(f"sequence {i} ({lens[i]} tokens): layer 31 + head rel logit err {err:.2e}")
        assert err <= LOGIT_TOL
    # end to end from the tokens: the shortest sequence through the pipeline
    # and then the merged worker (teacher-forced on the engine's tokens), the
    # longest through the pipeline
    i = int(np.argmin(lens))
    ow = OStage(cfg, W, 0, L)
    refs = [ow.prefill([0], [lens[i]], toks[starts[i]:starts[i + 1]])[-1]]
    refs += [ow.decode([0], np.array([fed[s][i]], np.int32))[0] for s in range(3)]
    got = [a_out[-1][i]] + [merged_logits[s][i] for s in range(3)]
    for s, (g_, r_) in enumerate(zip(got, refs)):
        err = np.abs(g_ - r_).max() / np.abs(r_).max()
        bound = logit_bound("c5_8b_full_shortest", s)
        say(f"shortest sequence ({lens[i]} tokens), "
            f"{'pipeline prefill' if s == 0 else f'merged decode step {s - 1}'}: "
            f"rel logit err {err:.2e} (bound {bound:.2e})")
        assert err <= bound
    j = int(np.argmax(lens))
    ref = OStage(cfg, W, 0, L).prefill([0], [lens[j]], toks[starts[j]:starts[j + 1]])[-1]
    err = np.abs(a_out[-1][j] - ref).max() / np.abs(ref).max()
    bound = logit_bound("c5_8b_full_longest", 0)
    say(f"longest sequence ({lens[j]} tokens): rel logit err {err:.2e} (bound {bound:.2e})")
    assert err <= bound
    del W
    gc.collect()
