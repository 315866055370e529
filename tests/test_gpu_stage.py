"""End-to-end parity of the stage engine on the tiny workload (2 layers, two
one-layer stages, 32-token prompt, 16 greedy decode steps), through the C ABI,
against the CPU oracle; plus the bitwise invariants and the error paths."""
import numpy as np
import pytest

import oracle
from oracle import kvblob
from oracle.llama import Stage as OStage, SyntheticWeights, greedy_generate
from workloads import WORKLOADS, gen
from tests import gpu_util as G

pytestmark = pytest.mark.gpu

WL = WORKLOADS["tiny-2x1"]
CFG = WL.cfg
LOGIT_TOL = 3e-2          # max |err| <= LOGIT_TOL * max |logit|


@pytest.fixture(scope="module")
def env():
    from paper_2502_15524_amd import hs, pipeline
    imgs = {}
    for rb, re in ((0, 2), (0, 1), (1, 2)):
        imgs[(rb, re)] = pipeline.pinned_image(CFG, rb, re)
    W = SyntheticWeights(CFG)
    prompt = gen.tokens(CFG.vocab, 32, WL.seed)
    o_toks, o_logits = greedy_generate(CFG, W, prompt, WL.decode_steps, stages=list(WL.stages))
    return dict(hs=hs, pipeline=pipeline, imgs=imgs, W=W, prompt=prompt, o_toks=o_toks,
                o_logits=o_logits)


def assert_oracle_teacher_forced(env, prompt, fed, gpu_logits):
    """The oracle (whole model, float32) on the prompt and then on the tokens
    the engine fed back, one decode step each: every row of the engine's
    logits (prefill's last position, then each step) within LOGIT_TOL of the
    largest oracle logit."""
    ost = OStage(CFG, env["W"], 0, CFG.n_layers)
    ref = [ost.prefill([0], [len(prompt)], np.asarray(prompt))[-1]]
    for t in fed:
        ref.append(ost.decode([0], np.array([t], np.int32))[0])
    ref = np.stack(ref)
    got = np.asarray(gpu_logits)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    err = np.abs(got - ref).max(axis=1) / np.abs(ref).max(axis=1)
    assert err.max() <= LOGIT_TOL, err


def make(env, begin, end, resident=None, load=True, **kw):
    rb, re = resident or (begin, end)
    opts = dict(max_seqs=8, max_ctx=640, max_batch_tokens=1024)
    opts.update(kw)
    st = env["pipeline"].Stage(CFG, begin, end, resident=(rb, re), **opts)
    if load:
        st.load(env["imgs"][(rb, re)], chunk_bytes=1 << 18)
    return st


def run_greedy(stages, prompt, n_steps, seq_id=0):
    """Prefill then greedy decode through stages in order; returns tokens and
    the logits of every step (float32, host)."""
    torch = G.torch()
    sp = G.stream_ptr()
    T = len(prompt)
    x = torch.from_numpy(np.asarray(prompt, np.int32)).cuda()
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    logits = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
    toks, lgs = [], []
    for st in stages:
        if st.end == CFG.n_layers:
            st.prefill([seq_id], [T], x.data_ptr(), nxt.data_ptr(), logits.data_ptr(), sp)
        else:
            out = torch.zeros((T, CFG.hidden), dtype=torch.bfloat16, device="cuda")
            st.prefill([seq_id], [T], x.data_ptr(), out.data_ptr(), 0, sp)
            x = out
    toks.append(int(nxt.item()))
    lgs.append(logits.cpu().numpy()[0].copy())
    for _ in range(n_steps):
        x = nxt.clone()
        for st in stages:
            if st.end == CFG.n_layers:
                st.decode([seq_id], x.data_ptr(), nxt.data_ptr(), logits.data_ptr(), sp)
            else:
                out = torch.zeros((1, CFG.hidden), dtype=torch.bfloat16, device="cuda")
                st.decode([seq_id], x.data_ptr(), out.data_ptr(), 0, sp)
                x = out
        toks.append(int(nxt.item()))
        lgs.append(logits.cpu().numpy()[0].copy())
    return np.array(toks, np.int32), np.stack(lgs)


def test_tiny_pipeline_matches_oracle(env):
    s0, s1 = make(env, 0, 1), make(env, 1, 2)
    toks, lgs = run_greedy([s0, s1], env["prompt"], WL.decode_steps)
    ol = env["o_logits"]
    err = np.abs(lgs - ol).max(axis=1) / np.abs(ol).max(axis=1)
    srt = np.sort(ol, axis=1)
    margin = (srt[:, -1] - srt[:, -2]) / np.abs(ol).max(axis=1)
    print("per-step rel logit err", np.round(err, 4))
    print("per-step oracle top-1/top-2 margin", np.round(margin, 4))
    assert err.max() <= LOGIT_TOL
    assert np.array_equal(toks, env["o_toks"]), (toks, env["o_toks"])


def test_split_equals_full_bitwise(env):
    s0, s1 = make(env, 0, 1), make(env, 1, 2)
    t_pipe, l_pipe = run_greedy([s0, s1], env["prompt"], 6)
    full = make(env, 0, 2)
    t_full, l_full = run_greedy([full], env["prompt"], 6)
    assert np.array_equal(t_pipe, t_full)
    assert np.array_equal(l_pipe, l_full)


def _hidden_prefill(st, tokens, seq_id=0):
    torch = G.torch()
    x = torch.from_numpy(np.asarray(tokens, np.int32)).cuda()
    out = torch.zeros((len(tokens), CFG.hidden), dtype=torch.bfloat16, device="cuda")
    st.prefill([seq_id], [len(tokens)], x.data_ptr(), out.data_ptr(), 0, G.stream_ptr())
    return G.from_dev_bf16(out)


def test_stage_boundary_hidden_matches_oracle(env):
    st = make(env, 0, 1)
    got = _hidden_prefill(st, env["prompt"])
    ref = OStage(CFG, env["W"], 0, 1).prefill([0], [32], env["prompt"])
    assert G.rel_fro(got, ref) <= 1e-2


def test_causality_bitwise(env):
    st = make(env, 0, 1)
    t1 = gen.tokens(CFG.vocab, 100, 77)
    t2 = t1.copy()
    t2[70] = (t2[70] + 5) % CFG.vocab
    h1 = _hidden_prefill(st, t1, seq_id=1)
    h2 = _hidden_prefill(st, t2, seq_id=2)
    assert np.array_equal(h1[:70], h2[:70])
    assert not np.array_equal(h1[70], h2[70])


def test_prefill_then_decode_close_to_recompute(env):
    full = make(env, 0, 2)
    toks, lgs = run_greedy([full], env["prompt"], 8, seq_id=3)
    seq = np.concatenate([env["prompt"], toks[:-1]]).astype(np.int32)
    fresh = make(env, 0, 2)
    # logits of every extended position via prefills of growing prefixes
    for k in (0, 4, 8):
        n = len(env["prompt"]) + k
        _, lf = run_greedy([fresh], seq[:n], 0, seq_id=100 + k)
        assert np.abs(lf[0] - lgs[k]).max() <= LOGIT_TOL * np.abs(lgs[k]).max()


def test_ragged_batch_prefill_and_decode(env):
    """Several sequences in one call (ragged, some longer than one decode
    split) against the oracle, sequence by sequence."""
    torch = G.torch()
    sp = G.stream_ptr()
    lens = [1, 17, 300, 530]
    ids = [11, 12, 13, 14]
    prompts = [gen.tokens(CFG.vocab, n, 40 + i) for i, n in enumerate(lens)]
    full = make(env, 0, 2)
    x = torch.from_numpy(np.concatenate(prompts).astype(np.int32)).cuda()
    nxt = torch.zeros(len(ids), dtype=torch.int32, device="cuda")
    logits = torch.zeros((len(ids), CFG.vocab), dtype=torch.float32, device="cuda")
    full.prefill(ids, lens, x.data_ptr(), nxt.data_ptr(), logits.data_ptr(), sp)
    got = [logits.cpu().numpy().copy()]
    for _ in range(3):
        inp = nxt.clone()
        full.decode(ids, inp.data_ptr(), nxt.data_ptr(), logits.data_ptr(), sp)
        got.append(logits.cpu().numpy().copy())
    # teacher-forced oracle on the engine's own tokens
    for i, (sid, p) in enumerate(zip(ids, prompts)):
        ost = OStage(CFG, env["W"], 0, 2)
        ref = [ost.prefill([sid], [len(p)], p)[-1]]
        cur = int(np.argmax(got[0][i]))
        for step in range(3):
            ref.append(ost.decode([sid], np.array([cur]))[0])
            cur = int(np.argmax(got[step + 1][i]))
        for step in range(4):
            r = ref[step]
            assert np.abs(got[step][i] - r).max() <= LOGIT_TOL * np.abs(r).max(), (sid, step)


def _export(st, ids):
    torch = G.torch()
    hs = st_hs()
    n = hs.hs_kv_export_size(st.h, ids)
    buf = torch.zeros(n, dtype=torch.uint8, device="cuda")
    w = hs.hs_kv_export(st.h, ids, buf.data_ptr(), n, G.stream_ptr())
    assert w == n
    return buf


def st_hs():
    from paper_2502_15524_amd import hs
    return hs


def test_kv_export_import_roundtrip_bitwise(env):
    hs = env["hs"]
    s0 = make(env, 0, 1)
    _hidden_prefill(s0, env["prompt"], seq_id=5)
    _hidden_prefill(s0, gen.tokens(CFG.vocab, 50, 9), seq_id=6)
    blob = _export(s0, [6, 5])
    b1 = blob.cpu().numpy().tobytes()
    hdr, seqs = kvblob.parse(b1)          # the oracle's codec reads it
    assert hdr["records"] == [(6, 50, 4), (5, 32, 2)]
    # logical K/V content against the oracle's cache
    ost = OStage(CFG, env["W"], 0, 1)
    ost.prefill([5], [32], env["prompt"])
    K, V = ost.kv[5][0]
    k_gpu = gen.bf16_bits_to_f32(seqs[1][1][0])
    v_gpu = gen.bf16_bits_to_f32(seqs[1][2][0])
    assert np.abs(k_gpu - K).max() <= 2e-2 * np.abs(K).max()
    assert np.abs(v_gpu - V).max() <= 2e-2 * np.abs(V).max()
    # import into a fresh stage, export again: identical bytes
    s0b = make(env, 0, 1)
    hs.hs_kv_import(s0b.h, blob.data_ptr(), blob.numel(), G.stream_ptr())
    assert hs.hs_seq_tokens(s0b.h, 5) == 32 and hs.hs_seq_tokens(s0b.h, 6) == 50
    b2 = _export(s0b, [6, 5]).cpu().numpy().tobytes()
    assert b1 == b2


def test_kv_roundtrip_many_sequences_bitwise(env):
    """A blob with more sequence records than the importer reads with the
    header in its first copy (300 sequences of 1-40 tokens)."""
    torch = G.torch()
    hs = env["hs"]
    n = 300
    lens = [int(x) for x in np.random.default_rng(300).integers(1, 41, n)]
    ids = list(range(1000, 1000 + n))
    toks = gen.tokens(CFG.vocab, sum(lens), 31)
    src = make(env, 0, 1, max_seqs=n, max_ctx=64, max_batch_tokens=sum(lens))
    x = torch.from_numpy(np.asarray(toks, np.int32)).cuda()
    out = torch.zeros((sum(lens), CFG.hidden), dtype=torch.bfloat16, device="cuda")
    src.prefill(ids, lens, x.data_ptr(), out.data_ptr(), 0, G.stream_ptr())
    order = ids[::-1]
    blob = _export(src, order)
    b1 = blob.cpu().numpy().tobytes()
    hdr, _ = kvblob.parse(b1)
    assert len(hdr["records"]) == n
    dst = make(env, 0, 1, max_seqs=n, max_ctx=64, max_batch_tokens=sum(lens))
    hs.hs_kv_import(dst.h, blob.data_ptr(), blob.numel(), G.stream_ptr())
    for i, ln in zip(ids, lens):
        assert hs.hs_seq_tokens(dst.h, i) == ln
    assert _export(dst, order).cpu().numpy().tobytes() == b1


def test_import_then_continue_decoding_bitwise(env):
    """Checkpoint/resume: a stage rebuilt from a blob decodes exactly like
    the original."""
    torch = G.torch()
    hs = env["hs"]
    full = make(env, 0, 2)
    t_ref, l_ref = run_greedy([full], env["prompt"], 0, seq_id=7)
    blob = _export(full, [7])
    fresh = make(env, 0, 2)
    hs.hs_kv_import(fresh.h, blob.data_ptr(), blob.numel(), G.stream_ptr())
    sp = G.stream_ptr()
    outs = []
    for st in (full, fresh):
        nxt = torch.tensor([int(t_ref[0])], dtype=torch.int32, device="cuda")
        lg = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
        seq = []
        for _ in range(4):
            inp = nxt.clone()
            st.decode([7], inp.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
            seq.append(lg.cpu().numpy().copy())
        outs.append(np.stack(seq))
    assert np.array_equal(outs[0], outs[1])


def test_merge_equals_pipeline_bitwise(env):
    hs = env["hs"]
    a0, a1 = make(env, 0, 1), make(env, 1, 2)
    b0, b1 = make(env, 0, 1), make(env, 1, 2)
    ta, la = run_greedy([a0, a1], env["prompt"], 2, seq_id=1)
    tb, lb = run_greedy([b0, b1], env["prompt"], 2, seq_id=1)
    assert np.array_equal(la, lb)
    merged = make(env, 0, 0, resident=(0, 2))
    hs.hs_stage_merge(merged.h, [b0.h, b1.h], G.stream_ptr())
    info = merged.info()
    assert (info["layer_begin"], info["layer_end"]) == (0, 2) and info["live_seqs"] == 1
    assert b0.info()["live_seqs"] == 0 and b1.info()["live_seqs"] == 0
    # continue both from the same token
    torch = G.torch()
    sp = G.stream_ptr()
    res, fed = [], []
    for stages in ([a0, a1], [merged]):
        nxt = torch.tensor([int(ta[-1])], dtype=torch.int32, device="cuda")
        lg = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
        seq = []
        fed = []
        for _ in range(5):
            fed.append(int(nxt.item()))
            x = nxt.clone()
            for st in stages:
                if st.end == CFG.n_layers:
                    st.decode([1], x.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
                else:
                    out = torch.zeros((1, CFG.hidden), dtype=torch.bfloat16, device="cuda")
                    st.decode([1], x.data_ptr(), out.data_ptr(), 0, sp)
                    x = out
            seq.append(lg.cpu().numpy().copy())
        res.append(np.stack(seq))
    assert np.array_equal(res[0], res[1])
    # and the merged worker against the oracle, fed the same tokens
    assert_oracle_teacher_forced(env, env["prompt"], list(ta[:2]) + fed,
                                 np.concatenate([lb, res[1][:, 0]]))


def test_import_many_equals_one_stage_and_decodes_bitwise(env):
    """The two one-layer stages' blobs of a sequence, imported in one call
    (hs_kv_import_many, headers handed over on the host) into a fresh
    two-layer stage: its export equals that of a two-layer stage that ran
    the prefill itself, byte for byte, and it decodes exactly like the
    pipeline. A bad blob anywhere in the list changes nothing."""
    torch = G.torch()
    hs = env["hs"]
    sp = G.stream_ptr()
    s0, s1 = make(env, 0, 1), make(env, 1, 2)
    toks, _ = run_greedy([s0, s1], env["prompt"], 1, seq_id=3)
    full = make(env, 0, 2)
    run_greedy([full], env["prompt"], 1, seq_id=3)
    blobs = []
    for st in (s0, s1):
        b = _export(st, [3])
        head = hs.hs_kv_export_head(st.h, [3])
        assert bytes(b[:len(head)].cpu().numpy().tobytes()) == head
        blobs.append((b, head))
    tgt = make(env, 0, 2)
    before = tgt.info()
    bad = blobs[1][0].clone()
    with pytest.raises(hs.HSError) as e:      # second blob's length disagrees with its head
        hs.hs_kv_import_many(tgt.h, [(blobs[0][0].data_ptr(), blobs[0][0].numel(), blobs[0][1]),
                                     (bad.data_ptr(), bad.numel() - 16, blobs[1][1])], sp)
    assert e.value.code == hs.HS_EINVAL and tgt.info() == before
    hs.hs_kv_import_many(tgt.h, [(b.data_ptr(), b.numel(), hd) for b, hd in blobs], sp)
    assert tgt.info()["live_seqs"] == 1 and hs.hs_seq_tokens(tgt.h, 3) == len(env["prompt"]) + 1
    assert _export(tgt, [3]).cpu().numpy().tobytes() == _export(full, [3]).cpu().numpy().tobytes()
    outs = []
    for stages in ([s0, s1], [tgt]):
        nxt = torch.tensor([int(toks[-1])], dtype=torch.int32, device="cuda")
        lg = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
        seq = []
        for _ in range(3):
            x = nxt.clone()
            for st in stages:
                if st.end == CFG.n_layers:
                    st.decode([3], x.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
                else:
                    o = torch.zeros((1, CFG.hidden), dtype=torch.bfloat16, device="cuda")
                    st.decode([3], x.data_ptr(), o.data_ptr(), 0, sp)
                    x = o
            seq.append(lg.cpu().numpy().copy())
        outs.append(np.stack(seq))
    assert np.array_equal(outs[0], outs[1])


def test_chunk_order_does_not_change_results(env):
    torch = G.torch()
    img = env["imgs"][(0, 2)]
    ref_st = make(env, 0, 2)
    _, l_ref = run_greedy([ref_st], env["prompt"], 2, seq_id=0)
    st = make(env, 0, 2, load=False)
    n_chunks = (img.numel() + (1 << 16) - 1) >> 16
    order = np.random.default_rng(3).permutation(n_chunks)
    st.load(img, chunk_bytes=1 << 16, order=list(order))
    _, l = run_greedy([st], env["prompt"], 2, seq_id=0)
    assert np.array_equal(l, l_ref)
    assert env["hs"].hs_stage_loaded(st.h) == (2, img.numel())


def test_error_paths(env):
    torch = G.torch()
    hs = env["hs"]
    sp = G.stream_ptr()
    x = torch.from_numpy(env["prompt"].astype(np.int32)).cuda()
    out = torch.zeros((32, CFG.hidden), dtype=torch.bfloat16, device="cuda")

    def code(f, *a):
        with pytest.raises(hs.HSError) as e:
            f(*a)
        return e.value.code

    st = make(env, 0, 1, load=False)
    assert code(st.prefill, [0], [32], x.data_ptr(), out.data_ptr(), 0, sp) == hs.HS_ENOTREADY
    img = env["imgs"][(0, 1)]
    descs, _ = hs.hs_weight_layout(st.c, 0, 1)
    layer0 = [d for d in descs if d["layer"] == 0]
    # only the embedding and half of layer 0: still not ready
    half = (layer0[0]["offset"] + layer0[-1]["offset"]) // 2
    hs.hs_stage_load_chunk(st.h, 0, img.data_ptr(), half)
    assert code(st.prefill, [0], [32], x.data_ptr(), out.data_ptr(), 0, sp) == hs.HS_ENOTREADY
    assert st.info()["live_seqs"] == 0
    # overlapping chunk rejected
    assert code(hs.hs_stage_load_chunk, st.h, 256, img.data_ptr() + 256, 1024) == hs.HS_EINVAL
    hs.hs_stage_load_chunk(st.h, half, img.data_ptr() + half, img.numel() - half)
    st.prefill([0], [32], x.data_ptr(), out.data_ptr(), 0, sp)
    # duplicate id, unknown id, too long
    assert code(st.prefill, [0], [32], x.data_ptr(), out.data_ptr(), 0, sp) == hs.HS_EINVAL
    one = torch.zeros(1, dtype=torch.int32, device="cuda")
    o1 = torch.zeros((1, CFG.hidden), dtype=torch.bfloat16, device="cuda")
    assert code(st.decode, [99], one.data_ptr(), o1.data_ptr(), 0, sp) == hs.HS_EINVAL
    small = make(env, 0, 1, max_ctx=33)
    small.prefill([0], [32], x.data_ptr(), out.data_ptr(), 0, sp)
    small.decode([0], one.data_ptr(), o1.data_ptr(), 0, sp)
    assert code(small.decode, [0], one.data_ptr(), o1.data_ptr(), 0, sp) == hs.HS_ERANGE
    # export into a too-small buffer reports the size
    need = hs.hs_kv_export_size(st.h, [0])
    tiny = torch.zeros(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(hs.HSError) as e:
        hs.hs_kv_export(st.h, [0], tiny.data_ptr(), 64, sp)
    assert e.value.code == hs.HS_ERANGE and e.value.required == need
    # host destination rejected
    hbuf = torch.zeros(need, dtype=torch.uint8)
    assert code(hs.hs_kv_export, st.h, [0], hbuf.data_ptr(), need, sp) == hs.HS_EINVAL
    # corrupted blob leaves the target unchanged
    blob = _export(st, [0])
    tgt = make(env, 0, 1)
    before = tgt.info()
    bad = blob.clone()
    bad[0] = 0
    assert code(hs.hs_kv_import, tgt.h, bad.data_ptr(), bad.numel(), sp) == hs.HS_EINVAL
    assert code(hs.hs_kv_import, tgt.h, blob.data_ptr(), blob.numel() - 16, sp) == hs.HS_EINVAL
    assert tgt.info() == before
    # blob layers not resident in the target
    other = make(env, 1, 2)
    assert code(hs.hs_kv_import, other.h, blob.data_ptr(), blob.numel(), sp) == hs.HS_EINVAL
    # not enough blocks: nothing is written
    cramped = make(env, 0, 1, kv_num_blocks=1)
    assert code(hs.hs_kv_import, cramped.h, blob.data_ptr(), blob.numel(), sp) == hs.HS_ENOMEM
    assert cramped.info()["live_seqs"] == 0 and cramped.info()["free_blocks"] == 1
    # a prefill or decode that cannot get its blocks changes nothing either
    assert code(cramped.prefill, [5], [32], x.data_ptr(), out.data_ptr(), 0, sp) == hs.HS_ENOMEM
    assert cramped.info()["live_seqs"] == 0 and cramped.info()["free_blocks"] == 1
    cramped.prefill([6], [16], x.data_ptr(), out.data_ptr(), 0, sp)     # one full block
    assert cramped.info()["free_blocks"] == 0
    assert code(cramped.decode, [6], one.data_ptr(), o1.data_ptr(), 0, sp) == hs.HS_ENOMEM
    assert hs.hs_seq_tokens(cramped.h, 6) == 16 and cramped.info()["free_blocks"] == 0
    # merge preconditions
    m = make(env, 0, 0, resident=(0, 2))
    s1 = make(env, 1, 2)
    assert code(hs.hs_stage_merge, m.h, [st.h, s1.h], sp) == hs.HS_ESTATE  # different sequences
    gap = make(env, 0, 0, resident=(0, 1))
    assert code(hs.hs_stage_merge, gap.h, [st.h, s1.h], sp) == hs.HS_ESTATE  # not resident
    assert st.info()["live_seqs"] == 1


def test_timing_sites_filter(env):
    """Timing every site reports every kernel of the forward pass; naming
    sites reports only their launches (one per layer, or one layer's with
    "site@layer"), and results do not depend on timing."""
    hs = env["hs"]
    st = make(env, 0, 2)
    hs.hs_stage_read_timing(st.h)
    hs.hs_stage_set_timing(st.h, 1)
    h_all = _hidden_prefill_full(st, env["prompt"], seq_id=1)
    all_stats = hs.hs_stage_read_timing(st.h)
    sites = {s["site"] for s in all_stats}
    assert {"embed", "attn_norm", "qkv", "attn", "o_proj", "ffn_norm", "gate_up",
            "down", "final_norm", "lm_head", "argmax"} <= sites
    hs.hs_stage_set_timing_sites(st.h, "qkv, down")
    h_two = _hidden_prefill_full(st, env["prompt"], seq_id=2)
    two = hs.hs_stage_read_timing(st.h)
    assert {s["site"] for s in two} == {"qkv", "down"}
    assert all(s["launches"] == CFG.n_layers and s["total_ms"] > 0 for s in two)
    # "site@layer" names one layer's launch; a layer outside the stage names none
    hs.hs_stage_set_timing_sites(st.h, "gate_up@1,qkv@7,lm_head@1")
    h_one = _hidden_prefill_full(st, env["prompt"], seq_id=3)
    one = hs.hs_stage_read_timing(st.h)
    assert [(s["site"], s["launches"]) for s in one] == [("gate_up", 1)]
    hs.hs_stage_set_timing(st.h, 0)
    hs.hs_stage_set_timing_sites(st.h, None)
    assert np.array_equal(h_all, h_two) and np.array_equal(h_all, h_one)


def _hidden_prefill_full(st, tokens, seq_id):
    torch = G.torch()
    x = torch.from_numpy(np.asarray(tokens, np.int32)).cuda()
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    logits = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
    st.prefill([seq_id], [len(tokens)], x.data_ptr(), nxt.data_ptr(), logits.data_ptr(),
               G.stream_ptr())
    return logits.cpu().numpy()


def test_scale_down_background_load_then_merge(env):
    """Scaling down: stage 0 serves layer 0 with memory for both layers and
    only layer 0's bytes loaded; it loads layer 1 (and the head) while the
    two-stage pipeline keeps decoding, then absorbs stage 1's KV cache and
    decodes alone. Tokens and logits equal an uninterrupted pipeline's,
    bitwise."""
    hs = env["hs"]
    torch = G.torch()
    sp = G.stream_ptr()
    ref_toks, ref_lgs = run_greedy([make(env, 0, 1), make(env, 1, 2)], env["prompt"], 9,
                                   seq_id=4)
    c = env["pipeline"].hs_cfg(CFG)
    descs, nbytes = hs.hs_weight_layout(c, 0, 2)
    first_end = max(d["offset"] + d["bytes"] for d in descs
                    if 0 <= d["layer"] < 1 or d["kind"] == hs.HS_W_EMBED)
    assert 0 < first_end < nbytes
    img = env["imgs"][(0, 2)]
    s0 = make(env, 0, 1, resident=(0, 2), load=False)
    hs.hs_stage_load_chunk(s0.h, 0, img.data_ptr(), first_end)
    s1 = make(env, 1, 2)
    assert hs.hs_stage_loaded(s0.h)[0] >= 1

    T = len(env["prompt"])
    x = torch.from_numpy(np.asarray(env["prompt"], np.int32)).cuda()
    hid = torch.zeros((T, CFG.hidden), dtype=torch.bfloat16, device="cuda")
    nxt = torch.zeros(1, dtype=torch.int32, device="cuda")
    lg = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
    s0.prefill([4], [T], x.data_ptr(), hid.data_ptr(), 0, sp)
    s1.prefill([4], [T], hid.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
    toks, lgs = [int(nxt.item())], [lg.cpu().numpy()[0].copy()]

    def decode(stages):
        xi = nxt.clone()
        for st in stages:
            if st.end == CFG.n_layers:
                st.decode([4], xi.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
            else:
                out = torch.zeros((1, CFG.hidden), dtype=torch.bfloat16, device="cuda")
                st.decode([4], xi.data_ptr(), out.data_ptr(), 0, sp)
                xi = out
        toks.append(int(nxt.item()))
        lgs.append(lg.cpu().numpy()[0].copy())

    for _ in range(3):
        decode([s0, s1])
    step = 4096
    for off in range(first_end, nbytes, step):       # background load, small chunks
        hs.hs_stage_load_chunk(s0.h, off, img.data_ptr() + off, min(step, nbytes - off))
    for _ in range(3):
        decode([s0, s1])                              # while the chunks land
    s0.sync()
    assert hs.hs_stage_loaded(s0.h) == (2, nbytes)
    hs.hs_stage_merge(s0.h, [s1.h], sp)
    assert (s0.begin, s0.end) == (0, 2) and s1.info()["live_seqs"] == 0
    for _ in range(3):
        decode([s0])
    assert np.array_equal(np.array(toks, np.int32), ref_toks)
    assert np.array_equal(np.stack(lgs), ref_lgs)
    assert_oracle_teacher_forced(env, env["prompt"], toks[:-1], np.stack(lgs))


def test_host_staged_migration_bitwise(env):
    """Host-staged migration: the blob written to pinned host memory chunk by
    chunk equals the device export byte for byte, its progress reaches the
    whole blob, and a stage that imports it from host memory (chunked) decodes
    exactly like the original."""
    torch = G.torch()
    hs = env["hs"]
    sp = G.stream_ptr()
    full = make(env, 0, 2)
    t_ref, _ = run_greedy([full], env["prompt"], 0, seq_id=8)
    dev_blob = _export(full, [8]).cpu().numpy().tobytes()
    size = len(dev_blob)
    host = torch.zeros(size + 64, dtype=torch.uint8).pin_memory()
    unit = 2 * 2 * CFG.n_kv_heads * 16 * CFG.head_dim      # one KV unit: K and V blocks
    for chunk in (unit, 3 * unit + 5, 1 << 30):
        host.zero_()
        n = hs.hs_kv_export_host(full.h, [8], host.data_ptr(), size + 64, chunk, sp)
        assert n == size
        full.sync()
        assert hs.hs_kv_host_progress(full.h) == size
        assert host[:size].numpy().tobytes() == dev_blob
    fresh = make(env, 0, 2)
    hs.hs_kv_import_host(fresh.h, host.data_ptr(), size, 2 * unit, sp)
    assert hs.hs_seq_tokens(fresh.h, 8) == len(env["prompt"])
    assert _export(fresh, [8]).cpu().numpy().tobytes() == dev_blob
    outs = []
    for st in (full, fresh):
        nxt = torch.tensor([int(t_ref[0])], dtype=torch.int32, device="cuda")
        lg = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
        seq = []
        for _ in range(4):
            inp = nxt.clone()
            st.decode([8], inp.data_ptr(), nxt.data_ptr(), lg.data_ptr(), sp)
            seq.append(lg.cpu().numpy().copy())
        outs.append(np.stack(seq))
    assert np.array_equal(outs[0], outs[1])
    size2 = hs.hs_kv_export_size(full.h, [8])     # the sequence grew while decoding
    dev = torch.zeros(size2, dtype=torch.uint8, device="cuda")
    with pytest.raises(hs.HSError) as e:       # device memory is not a host blob
        hs.hs_kv_export_host(full.h, [8], dev.data_ptr(), size2, unit, sp)
    assert e.value.code == hs.HS_EINVAL
    with pytest.raises(hs.HSError) as e:
        hs.hs_kv_export_host(full.h, [8], host.data_ptr(), size2 - 1, unit, sp)
    assert e.value.code == hs.HS_ERANGE and e.value.required == size2


def test_continuous_batching_then_merge_bitwise(env):
    """Sequences join (prefilled one per call) and leave between decode steps
    of a two-stage pipeline whose first stage can hold both layers; midway the
    pipeline is drained and merged into that stage. Every sequence's logits at
    every step equal those of the sequence decoded alone, bitwise (decode
    arithmetic is per row, so batch composition does not change the bits)."""
    hs = env["hs"]
    torch = G.torch()
    sp = G.stream_ptr()
    prompts = {11: env["prompt"], 12: gen.tokens(CFG.vocab, 40, 21),
               13: gen.tokens(CFG.vocab, 17, 22)}

    def alone(sid, n):
        toks, lgs = run_greedy([make(env, 0, 1), make(env, 1, 2)], prompts[sid], n, seq_id=sid)
        return lgs

    ref = {11: alone(11, 5), 12: alone(12, 6), 13: alone(13, 3)}
    s0 = make(env, 0, 1, resident=(0, 2))
    s1 = make(env, 1, 2)
    got = {sid: [] for sid in prompts}
    fed = {sid: [] for sid in prompts}
    nxt = {}

    def prefill(stages, sid):
        p = prompts[sid]
        T = len(p)
        x = torch.from_numpy(np.asarray(p, np.int32)).cuda()
        hid = torch.zeros((T, CFG.hidden), dtype=torch.bfloat16, device="cuda")
        tok = torch.zeros(1, dtype=torch.int32, device="cuda")
        lg = torch.zeros((1, CFG.vocab), dtype=torch.float32, device="cuda")
        stages[0].prefill([sid], [T], x.data_ptr(), hid.data_ptr(), 0, sp)
        stages[1].prefill([sid], [T], hid.data_ptr(), tok.data_ptr(), lg.data_ptr(), sp)
        nxt[sid] = int(tok.item())
        got[sid].append(lg.cpu().numpy()[0].copy())

    def decode(stages, ids):
        B = len(ids)
        for i in ids:
            fed[i].append(nxt[i])
        x = torch.tensor([nxt[i] for i in ids], dtype=torch.int32, device="cuda")
        tok = torch.zeros(B, dtype=torch.int32, device="cuda")
        lg = torch.zeros((B, CFG.vocab), dtype=torch.float32, device="cuda")
        for st in stages:
            if st.end == CFG.n_layers:
                st.decode(ids, x.data_ptr(), tok.data_ptr(), lg.data_ptr(), sp)
            else:
                out = torch.zeros((B, CFG.hidden), dtype=torch.bfloat16, device="cuda")
                st.decode(ids, x.data_ptr(), out.data_ptr(), 0, sp)
                x = out
        t, l = tok.cpu().numpy(), lg.cpu().numpy()
        for k, i in enumerate(ids):
            nxt[i] = int(t[k])
            got[i].append(l[k].copy())

    pipe = [s0, s1]
    prefill(pipe, 11)
    decode(pipe, [11])
    decode(pipe, [11])
    prefill(pipe, 12)                        # joins
    decode(pipe, [11, 12])
    decode(pipe, [12, 11])                   # order within a batch does not matter
    prefill(pipe, 13)                        # joins
    decode(pipe, [11, 12, 13])
    for st in pipe:                          # 11 leaves after its last step
        hs.hs_seq_free(st.h, 11)
    decode(pipe, [13, 12])
    hs.hs_stage_merge(s0.h, [s1.h], sp)      # drain and consolidate
    assert s0.info()["live_seqs"] == 2 and s1.info()["live_seqs"] == 0
    decode([s0], [12, 13])
    decode([s0], [12])                       # 13 finished; 12 runs on alone
    for sid, lgs in got.items():
        assert len(lgs) == len(ref[sid]), sid
        assert np.array_equal(np.stack(lgs), ref[sid]), sid
        assert_oracle_teacher_forced(env, prompts[sid], fed[sid], np.stack(lgs))
