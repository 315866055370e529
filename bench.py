"""Benchmark of the pipeline-stage engine on one MI355X.

Headline workload: the Llama-2-7B-shaped model cut into 4 stages; the second
stage (layers 8-15) serves one 512-token prompt (batch 1), fed the hidden
states that the first stage (layers 0-7, run on the GPU beforehand) computes
from the seeded prompt. One step is one prefill of that prompt through the
stage with its weights resident in HBM (the stage's contribution to TTFT);
`value` is prompt tokens per second over the K timed steps. Reported beside it:
  * cold TTFT: weights streamed from pinned host memory in chunks while the
    stage prefills (each layer starts when its bytes land), host wall clock
    from the first chunk enqueue to the output being ready (PCIe-inclusive),
    and the same including the stage's creation;
  * decode: batch-1 decode steps of the same stage (HBM-bound);
  * KV export / import of the stage's cache (device to device);
  * roofline of the dominant kernel, timed with HIP events on the launch
    stream inside the timed region;
  * the CPU oracle timed on this host on the same prefill (all threads and
    one thread, CPU model and BLAS named).
Then, unless --no-extras, the other full-size workloads as extra keys, each
with its own roofline and an oracle sample: the 7B model as one stage (batch
8 x 1024, 128 greedy decode steps with the tokens fed back), the 13B model's
first 20-layer stage loaded cold while it prefills 4 x 2048 tokens, and the
8B-GQA model in 4 stages (16 ragged prompts) whose KV caches are exported,
imported and merged into one worker that decodes 256 greedy steps.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-extras]
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6    # 256 CU x 2.4 GHz x 4096 flop/clk (dense)
PEAK_HBM_GBPS = 8000.0
PEAK_PCIE_GBPS = 64.0        # PCIe 5.0 x16, per direction
METRIC = ("cold TTFT (weights in host) ms; prefill tok/s; decode tok/s; "
          "% of MFMA/HBM peak")
EXTRAS = ("c3", "c4", "c5")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cold-runs", type=int, default=5)
    ap.add_argument("--decode-steps", type=int, default=64)
    ap.add_argument("--chunk-mb", type=int, default=64)
    ap.add_argument("--cold-chunk-mb", type=int, default=64,
                    help="chunk size of the 13B stage's cold load (extra c4)")
    ap.add_argument("--copy-streams", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--workload", default="7b-stage8-15-cold",
                    help="7b-stage8-15-cold (default: one stage, cold TTFT) or one of "
                         "7b-full-b8, 13b-2x20-b4, 8b-4x8-ragged-merge (whole pipeline on "
                         "this GPU: batched prefill, decode, and for the last one KV "
                         "export/import and merge), 13b-4x10-scale-down (per-token decode "
                         "times while the first stage loads the rest of the model in the "
                         "background, then merges the others)")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="only run a few warm prefill steps and a 256 MiB device copy "
                         "(the workload for hardware-counter passes)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 counter passes over a --traffic-probe run "
                         "(no GPU work)")
    ap.add_argument("--gemm-shapes", action="store_true",
                    help="time the projection GEMMs of the 7B and 8B-GQA shapes through the "
                         "kernel entry point beside torch.matmul (hipBLASLt) on the same "
                         "shapes; prints a markdown table")
    ap.add_argument("--no-extras", action="store_true",
                    help="headline workload only")
    ap.add_argument("--extras", default=",".join(EXTRAS),
                    help="comma list of the extra workloads to run after the headline: "
                         "c3 (7B full, batch 8), c4 (13B stage 0 cold), c5 (8B ragged, "
                         "KV migration and merge)")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _sha(path):
    """SHA-256 of a kernel source's code: comments and blank lines removed and
    runs of whitespace collapsed, so that a counter summary stays valid across
    edits of the text around the code but not across any change to it."""
    import re
    with open(path, encoding="utf-8") as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    lines = [" ".join(l.split()) for l in src.splitlines()]
    return hashlib.sha256("\n".join(l for l in lines if l).encode()).hexdigest()


def traffic_from_profiles(kernel, workload=None):
    """HBM bytes per launch of `kernel` from the committed counter summaries
    (profiles/*traffic*.md, lines "traffic: kernel=K [workload=W]
    hbm_bytes_per_launch=B <source>_sha256=H"), if they were taken on the
    current source of that kernel (k_gemm.hip, k_attn.hip or k_misc.hip);
    else None."""
    csrc = os.path.join(ROOT, "paper_2502_15524_amd", "csrc")
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*traffic*.md"))):
        with open(path) as f:
            for line in f:
                if not line.startswith("traffic:"):
                    continue
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                if kv.get("kernel") != kernel:
                    continue
                if workload is not None and kv.get("workload", workload) != workload:
                    continue
                src = [k for k in kv if k.endswith("_sha256")]
                if not src:
                    continue
                fname = src[0][:-len("_sha256")] + ".hip"
                if _sha(os.path.join(csrc, fname)) == kv[src[0]]:
                    return int(kv["hbm_bytes_per_launch"])
    return None


def host_info():
    """CPU model, logical CPUs and the BLAS numpy uses (threadpoolctl)."""
    from threadpoolctl import threadpool_info
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
    b = blas[0] if blas else {}
    return {"cpu_model": model, "host_cpus": os.cpu_count(),
            "blas": f"{b.get('internal_api', '?')} {b.get('version', '')}".strip(),
            "blas_threads": int(b.get("num_threads", 1))}


def oracle_timed(fn, min_seconds, threads=None):
    """Repeat fn() for at least min_seconds (BLAS limited to `threads` if
    given); returns (repetitions, seconds)."""
    from threadpoolctl import threadpool_limits
    reps, dt = 0, 0.0
    with threadpool_limits(limits=threads, user_api="blas"):
        while dt < min_seconds:
            t0 = time.perf_counter()
            fn(reps)
            dt += time.perf_counter() - t0
            reps += 1
    return reps, dt


def layer_weights(cfg, layers, threads=16):
    """The oracle's float32 weights of the given layers, drawn in parallel."""
    import concurrent.futures as cf
    from oracle.llama import SyntheticWeights
    W = SyntheticWeights(cfg)
    items = [(l, k) for l in layers for k in ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown")]
    with cf.ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda it: W(*it), items))
    return W


def cpu_baseline(wl, x_f32, stage_range, min_seconds=12.0):
    """The oracle, as it stands, on the same prefill (all 512 tokens, all 8
    layers of the stage), on this host's cores; then one layer of it with
    one BLAS thread."""
    from oracle.llama import Stage
    cfg = wl.cfg
    b, e = stage_range
    W = layer_weights(cfg, range(b, e))
    st = Stage(cfg, W, b, e)
    n = x_f32.shape[0]

    def run(i):
        st.prefill([i], [n], x_f32)
        st.drop(i)
    reps, dt = oracle_timed(run, min_seconds)
    one = Stage(cfg, W, b, b + 1)

    def run1(i):
        one.prefill([i], [n], x_f32)
        one.drop(i)
    reps1, dt1 = oracle_timed(run1, 3.0, threads=1)
    hi = host_info()
    res = {"value": round(reps * n / dt, 2), "unit": "tok/s", "cores": hi["blas_threads"],
           "kind": "oracle",
           "sample": f"{reps} full prefills of the {n}-token prompt through layers {b}-{e - 1} "
                     f"(numpy float32, {dt:.1f} s in total)",
           "value_1thread": round(reps1 * n / dt1 / (e - b), 2),
           "sample_1thread": f"{reps1} prefills of the prompt through layer {b} alone with one "
                             f"BLAS thread ({dt1:.1f} s), scaled to {e - b} layers"}
    res.update(hi)
    return res


def main():
    args = parse()
    if args.summarize_counters:
        return summarize_counters(*args.summarize_counters, workload=args.workload)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the stage engine "
              "has no multi-GPU path in this build", file=sys.stderr)
        sys.exit(2)
    # The weight upload overlaps the prefill only if the stage's copy streams
    # do not share a hardware queue with the stream the prefill runs on (a
    # shared queue runs the prefill after every copy queued before it). HIP
    # spreads streams over GPU_MAX_HW_QUEUES queues (4 by default); with the
    # benchmark's streams plus two copy streams per stage, 8 keeps them apart.
    # It must be set before the HIP runtime starts.
    os.environ["GPU_MAX_HW_QUEUES"] = os.environ.get("HS_BENCH_HW_QUEUES", "8")
    import torch
    from workloads import WORKLOADS

    assert torch.cuda.is_available()
    if args.gemm_shapes:
        return gemm_shapes()
    if args.workload.endswith("scale-down"):
        res = bench_scale_down(WORKLOADS[args.workload], args)
    elif args.workload != "7b-stage8-15-cold":
        res = bench_pipeline(WORKLOADS[args.workload], args)
    else:
        res = bench_c2(args)
        if res is not None and not args.no_extras:
            want = [x for x in args.extras.split(",") if x]
            if "c3" in want:
                res["c3_7b_full_b8"] = bench_pipeline(WORKLOADS["7b-full-b8"], args,
                                                      n_dec=128, oracle_sample=True)
            if "c4" in want:
                res["c4_13b_stage0_cold"] = bench_cold_stage(WORKLOADS["13b-2x20-b4"], args)
            if "c5" in want:
                res["c5_8b_ragged_merge"] = bench_pipeline(
                    WORKLOADS["8b-4x8-ragged-merge"], args, n_dec=256, oracle_sample=True)
    if res is not None:
        print(json.dumps(res), flush=True)


def gemm_shapes(reps=20, copies=4):
    """The decoder-layer projections of the 7B shape at 512 and 8192 prompt
    tokens and at 1 and 8 decode tokens, and of the 8B-GQA shape at 16 decode
    tokens, each timed with HIP events over `reps` launches through
    hs_k_gemm (the library picks the configuration as in a stage) with
    `copies` weight matrices in rotation, so the weights stream from HBM as in
    a stage; beside them torch.matmul (hipBLASLt) of the same operands, which
    writes the plain product (no residual read, no SwiGLU halving). Random
    bf16 operands (timing only). QKV runs with the plain-store epilogue here;
    in a stage, prompts of more than 64 tokens rotate and append in the QKV
    epilogue and decode batches fold the RMSNorm into QKV and gate/up."""
    import torch
    from paper_2502_15524_amd import hs
    from workloads import MODELS
    dev = "cuda"
    rows = []
    for model, Ms in (("llama2-7b", (512, 8192, 1, 8)), ("llama3-8b", (16,))):
        cfg = MODELS[model]
        H, F, D = cfg.hidden, cfg.ffn, cfg.head_dim
        projs = (("qkv", (cfg.n_heads + 2 * cfg.n_kv_heads) * D, H, 0),
                 ("o", H, cfg.n_heads * D, 1), ("gate/up", 2 * F, H, 2), ("down", H, F, 1))
        for M in Ms:
            for name, N, K, epi in projs:
                kp = (K + 63) // 64 * 64
                X = torch.zeros(M, kp, device=dev, dtype=torch.bfloat16)
                X[:, :K] = torch.randn(M, K, device=dev).bfloat16()
                Ws = [(torch.randn(N, K, device=dev) * 0.02).bfloat16() for _ in range(copies)]
                ncol = N // 2 if epi == 2 else N
                Y = torch.zeros(M, ncol, device=dev, dtype=torch.bfloat16)
                R = torch.randn(M, ncol, device=dev).bfloat16()
                it = [0]

                def ours():
                    W = Ws[it[0] % copies]
                    it[0] += 1
                    hs.hs_k_gemm(X.data_ptr(), kp, W.data_ptr(), Y.data_ptr(), ncol,
                                 R.data_ptr() if epi == 1 else 0, ncol, M, N, K, epi, 0)

                def theirs():
                    W = Ws[it[0] % copies]
                    it[0] += 1
                    torch.matmul(X[:, :K], W.t())

                res = []
                for fn in (ours, theirs):
                    for _ in range(3):
                        fn()
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    torch.cuda.synchronize()
                    e0.record()
                    for _ in range(reps):
                        fn()
                    e1.record()
                    torch.cuda.synchronize()
                    res.append(e0.elapsed_time(e1) / reps * 1e3)
                flops = 2.0 * M * N * K
                wbytes = 2.0 * N * K
                rows.append(f"| {model} | {M} | {name} | {N} x {K} | {res[0]:.1f} | "
                            f"{flops / res[0] / 1e6:.0f} | {wbytes / res[0] / 1e3:.0f} | "
                            f"{res[1]:.1f} | {flops / res[1] / 1e6:.0f} |")
                log(rows[-1])
                del Ws, X, Y, R
    print("| model | tokens | projection | N x K | hs_k_gemm us | TFLOP/s | weight GB/s | "
          "torch.matmul us | TFLOP/s |")
    print("|---|---|---|---|---|---|---|---|---|")
    for r in rows:
        print(r)
    return None


def bench_c2(args):
    """The headline workload (see the module docstring); returns the JSON
    line as a dict (None for --traffic-probe)."""
    import numpy as np
    import torch
    from paper_2502_15524_amd import hs, pipeline
    from workloads import WORKLOADS, gen

    wl = WORKLOADS["7b-stage8-15-cold"]
    cfg = wl.cfg
    b, e = wl.stages[wl.bench_stage]
    P = wl.prompt_lens[0]
    H = cfg.hidden
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()
    sp = stream.cuda_stream
    n_dec_in = args.decode_steps

    # The stage's input: the first stage (layers 0-7, with the embedding) run
    # on this GPU on the seeded prompt, and on one seeded token per decode
    # step (its decode outputs feed the middle stage's decode steps).
    t = time.perf_counter()
    img0 = pipeline.pinned_image(cfg, 0, b)
    first = pipeline.Stage(cfg, 0, b, max_seqs=1, max_ctx=P + n_dec_in + 8, max_batch_tokens=P)
    first.load(img0, 64 << 20)
    first.sync()
    img0.close()
    toks = torch.from_numpy(gen.tokens(cfg.vocab, P, wl.seed)).to(dev)
    x = torch.empty((P, H), dtype=torch.bfloat16, device=dev)
    first.prefill([0], [P], toks.data_ptr(), x.data_ptr(), 0, sp)
    dec_tok = torch.from_numpy(gen.tokens(cfg.vocab, n_dec_in, wl.seed + 100)).to(dev)
    xdec = torch.empty((n_dec_in, H), dtype=torch.bfloat16, device=dev)
    for k in range(n_dec_in):
        first.decode([0], dec_tok[k:k + 1].data_ptr(), xdec[k:k + 1].data_ptr(), 0, sp)
    stream.synchronize()
    first.close()
    log(f"[bench] stage input: layers 0-{b - 1} on the GPU ({P}-token prompt, {n_dec_in} decode "
        f"tokens) in {time.perf_counter() - t:.1f} s")
    x_f32 = x.float().cpu().numpy()

    t = time.perf_counter()
    img = pipeline.pinned_image(cfg, b, e)
    log(f"[bench] packed stage image {img.numel() / 1e9:.3f} GB in {time.perf_counter() - t:.1f} s")
    out = torch.empty((P, H), dtype=torch.bfloat16, device=dev)
    max_ctx = P + max(args.decode_steps, 9) + 16
    st = pipeline.Stage(cfg, b, e, max_seqs=4, max_ctx=max_ctx, max_batch_tokens=P,
                        n_copy_streams=args.copy_streams)
    chunk = args.chunk_mb << 20
    sid = [1000]

    def new_id():
        sid[0] += 1
        return sid[0]

    def prefill_once():
        i = new_id()
        st.prefill([i], [P], x.data_ptr(), out.data_ptr(), 0, sp)
        return i

    if args.traffic_probe:
        # Counter passes read FETCH_SIZE / WRITE_SIZE per dispatch; the plain
        # device-to-device copy of a known size calibrates them.
        st.load(img, chunk)
        st.sync()
        for _ in range(3):
            hs.hs_seq_free(st.h, prefill_once())
        i = prefill_once()
        od = torch.empty((1, H), dtype=torch.bfloat16, device=dev)
        for k in range(4):
            st.decode([i], xdec[k:k + 1].data_ptr(), od.data_ptr(), 0, sp)
        size = hs.hs_kv_export_size(st.h, [i])
        blob = torch.empty(size, dtype=torch.uint8, device=dev)
        head = hs.hs_kv_export_head(st.h, [i])
        dst = pipeline.Stage(cfg, b, e, max_seqs=4, max_ctx=max_ctx, max_batch_tokens=P)
        for _ in range(2):
            hs.hs_kv_export(st.h, [i], blob.data_ptr(), size, sp)
            hs.hs_kv_import_many(dst.h, [(blob.data_ptr(), size, head)], sp)
            stream.synchronize()
            hs.hs_seq_free(dst.h, i)
        dst.close()
        traffic_calibration_copies(torch, dev)
        log("[bench] traffic probe done: 3 prefill steps, 4 decode steps, 2 KV exports and "
            "imports, 2 copies of 268435456 bytes")
        st.close()
        return None

    # ---------------------------------------------------------- cold TTFT
    cold, load_only = [], []
    for r in range(args.cold_runs + 1):
        hs.hs_stage_invalidate_weights(st.h)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st.load(img, chunk)
        i = prefill_once()
        stream.synchronize()
        dt = time.perf_counter() - t0
        st.sync()
        hs.hs_seq_free(st.h, i)
        if r > 0:
            cold.append(dt)
        hs.hs_stage_invalidate_weights(st.h)
        t0 = time.perf_counter()
        st.load(img, chunk)
        st.sync()
        if r > 0:
            load_only.append(time.perf_counter() - t0)
    t_cold = statistics.median(cold)
    t_load = statistics.median(load_only)
    log(f"[bench] cold TTFT {t_cold * 1e3:.2f} ms, load only {t_load * 1e3:.2f} ms")
    # the same, including the creation of the stage (device memory for the
    # weights, KV pools and workspace, streams, events)
    with_create = []
    for r in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st2 = pipeline.Stage(cfg, b, e, max_seqs=4, max_ctx=max_ctx, max_batch_tokens=P,
                             n_copy_streams=args.copy_streams)
        st2.load(img, chunk)
        st2.prefill([1], [P], x.data_ptr(), out.data_ptr(), 0, sp)
        stream.synchronize()
        with_create.append(time.perf_counter() - t0)
        st2.close()
    t_cold_create = statistics.median(with_create)
    log(f"[bench] cold TTFT including hs_stage_create {t_cold_create * 1e3:.2f} ms")

    # -------------------------------------------------------- warm prefill
    # Warm-up steps run with every launch timed: they give the per-kernel
    # breakdown and name the dominant kernel. The timed steps then bracket
    # only that kernel's launch in the stage's middle layer with events
    # (events between back-to-back kernels cost time of their own; every
    # layer's launch has the same shape).
    def run_steps(k):
        ids = []
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        t0 = time.perf_counter()
        for _ in range(k):
            ids.append(prefill_once())
            if len(ids) >= 3:                # keep KV blocks bounded
                hs.hs_seq_free(st.h, ids.pop(0))
        ev1.record(stream)
        stream.synchronize()
        wall = time.perf_counter() - t0
        for i in ids:
            hs.hs_seq_free(st.h, i)
        return max(ev0.elapsed_time(ev1), wall * 1e3) / k

    hs.hs_stage_read_timing(st.h)            # reset counters
    hs.hs_stage_set_timing_sites(st.h, None)
    hs.hs_stage_set_timing(st.h, 1)
    run_steps(max(args.warmup, 1))
    hs.hs_stage_set_timing(st.h, 0)
    stats = hs.hs_stage_read_timing(st.h)
    nw = max(args.warmup, 1)
    kern_ms = sum(s["total_ms"] for s in stats)
    flops_step = sum(s["flops"] for s in stats) / nw
    log("[bench] warm-up steps with every launch timed:")
    for s in sorted(stats, key=lambda s: -s["total_ms"]):
        avg = s["total_ms"] / s["launches"]
        rate = (s["flops"] / s["launches"]) / (avg / 1e3) / 1e12 if s["flops"] else 0
        bw = (s["bytes"] / s["launches"]) / (avg / 1e3) / 1e9 if s["bytes"] else 0
        log(f"[bench]   {s['name']:<28} {s['site']:<10} x{s['launches'] // nw:<3} avg "
            f"{avg * 1e3:8.1f} us {100 * s['total_ms'] / kern_ms:5.1f}%  {rate:7.1f} TFLOP/s "
            f"{bw:7.0f} GB/s")
    dom = max(stats, key=lambda s: s["total_ms"])

    # the warm-up steps' per-launch events leave the next few steps slower
    # than steady state: settle with untimed steps before the timed region
    run_steps(max(args.warmup, 1))
    per_layer = dom["launches"] // nw == e - b
    hs.hs_stage_set_timing_sites(
        st.h, f"{dom['site']}@{(b + e) // 2}" if per_layer else dom["site"])
    hs.hs_stage_set_timing(st.h, 1)
    ms_step = run_steps(args.steps)
    hs.hs_stage_set_timing(st.h, 0)
    hs.hs_stage_set_timing_sites(st.h, None)
    timed = [s for s in hs.hs_stage_read_timing(st.h)
             if s["name"] == dom["name"] and s["site"] == dom["site"]]
    assert timed and timed[0]["launches"] == args.steps * (1 if per_layer else dom["launches"] // nw)
    dom = timed[0]
    tok_s = P / (ms_step / 1e3)
    t_prefill = ms_step / 1e3
    log(f"[bench] warm prefill {ms_step:.3f} ms/step = {tok_s:,.0f} tok/s "
        f"({flops_step / (ms_step / 1e3) / 1e12:.0f} TFLOP/s over the step)")
    ms_step_plain = run_steps(args.steps)
    log(f"[bench] same steps without any kernel events: {ms_step_plain:.3f} ms/step")
    dom_avg_s = dom["total_ms"] / dom["launches"] / 1e3
    dom_flops = dom["flops"] / dom["launches"]
    achieved = dom_flops / dom_avg_s / 1e12
    log(f"[bench] dominant kernel {dom['name']} ({dom['site']}"
        f"{f', layer {(b + e) // 2}' if per_layer else ''}): {dom_avg_s * 1e6:.1f} us, "
        f"{achieved:.0f} TFLOP/s in the timed steps")
    roofline = {"bound": "mfma", "kernel": dom["name"],
                "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic_from_profiles(dom["name"], wl.name),
                "flops_per_launch": dom_flops, "avg_launch_us": round(dom_avg_s * 1e6, 2)}
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)

    # ------------------------------------------------------------- decode
    # decode step k is fed the first stage's output for decode token k
    i = prefill_once()
    od = torch.empty((1, H), dtype=torch.bfloat16, device=dev)
    step = [0]

    def dec():
        k = step[0] % n_dec_in
        st.decode([i], xdec[k:k + 1].data_ptr(), od.data_ptr(), 0, sp)
        step[0] += 1
    for _ in range(4):
        dec()
    stream.synchronize()
    nd = max(args.decode_steps - 8, 1)
    ev0.record(stream)
    for _ in range(nd):
        dec()
    ev1.record(stream)
    stream.synchronize()
    dec_ms = ev0.elapsed_time(ev1) / nd

    def two_decode_steps():
        for _ in range(4):
            dec()
        stream.synchronize()
    dstats = log_decode_breakdown(hs, [st], two_decode_steps, 2)
    ctx = P + 4 + nd / 2.0
    kv_tok = 2 * cfg.n_kv_heads * cfg.head_dim * 2 * (e - b)
    dec_bytes = img.numel() + ctx * kv_tok
    log(f"[bench] decode B=1 {dec_ms:.3f} ms/step ({dec_bytes / (dec_ms / 1e3) / 1e9:.0f} GB/s)")

    # ------------------------------------------------------ KV export/import
    size = hs.hs_kv_export_size(st.h, [i])
    blob = torch.empty(size, dtype=torch.uint8, device=dev)
    hs.hs_kv_export(st.h, [i], blob.data_ptr(), size, sp)
    stream.synchronize()
    reps = 10
    ev0.record(stream)
    for _ in range(reps):
        hs.hs_kv_export(st.h, [i], blob.data_ptr(), size, sp)
    ev1.record(stream)
    stream.synchronize()
    exp_ms = ev0.elapsed_time(ev1) / reps
    dst = pipeline.Stage(cfg, b, e, max_seqs=4, max_ctx=max_ctx, max_batch_tokens=P)
    head = hs.hs_kv_export_head(st.h, [i])
    hs.hs_kv_import_many(dst.h, [(blob.data_ptr(), size, head)], sp)   # warm
    stream.synchronize()
    hs.hs_seq_free(dst.h, i)
    imp, imp1 = [], []
    for r in range(2 * reps):
        ev0.record(stream)
        if r % 2:       # header read back from the device blob
            hs.hs_kv_import(dst.h, blob.data_ptr(), size, sp)
        else:           # header handed over by the exporter
            hs.hs_kv_import_many(dst.h, [(blob.data_ptr(), size, head)], sp)
        ev1.record(stream)
        stream.synchronize()
        (imp1 if r % 2 else imp).append(ev0.elapsed_time(ev1))
        hs.hs_seq_free(dst.h, i)
    imp_ms = statistics.median(imp)
    used = size - len(head)
    log(f"[bench] KV export {2 * used / (exp_ms / 1e3) / 1e9:.0f} GB/s, "
        f"import {2 * used / (imp_ms / 1e3) / 1e9:.0f} GB/s ({used / 1e6:.1f} MB)")
    dst.close()

    # Equation 1 of the TTFT model for this stage as one full-memory worker
    # whose weights are already in host memory (no network fetch, no
    # initialisation): load the image at the measured host-link rate, then
    # prefill. The engine overlaps the two layer by layer, so it beats this.
    from paper_2502_15524_amd.controller import History, Server, predict_ttft
    h_rate = img.numel() / t_load
    ttft_eq1 = predict_ttft(History(t_c=0.0, t_n=0.0, t_p=t_prefill, t_d=dec_ms / 1e3),
                            img.numel(), 1, 1, [Server("local", float("inf"), h_rate, 1e12)])
    log(f"[bench] cold TTFT {t_cold * 1e3:.2f} ms measured vs {ttft_eq1 * 1e3:.2f} ms from "
        f"equation 1 (load {img.numel() / h_rate * 1e3:.2f} ms, then prefill)")

    base = None
    if not args.no_cpu_baseline:
        base = cpu_baseline(wl, x_f32, (b, e))
        log(f"[bench] oracle on host: {base['value']} tok/s with {base['cores']} threads")

    res = {
        "metric": METRIC, "value": round(tok_s, 1), "unit": "tok/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "shape": "llama2-7b (32 layers, hidden 4096, 32x128 "
                   "heads, ffn 11008)", "stage_layers": [b, e - 1], "batch": 1,
                   "prompt_len": P, "weights": "N(0,0.02) bf16, seeded"},
        "roofline": roofline,
        "cpu_baseline": base,
        "ms_per_step_without_kernel_events": round(ms_step_plain, 4),
        "timed_site": dom["site"],
        "prefill_mfma_frac_step": round(flops_step / t_prefill / 1e12 / PEAK_BF16_TFLOPS, 4),
        "input": f"hidden states of layers 0-{b - 1} computed on the GPU from the seeded prompt",
        "cold_ttft_ms": round(t_cold * 1e3, 3),
        "cold_ttft_with_create_ms": round(t_cold_create * 1e3, 3),
        "cold_ttft_predicted_eq1_ms": round(ttft_eq1 * 1e3, 3),
        "cold_load_only_ms": round(t_load * 1e3, 3),
        "h2d_GBps": round(img.numel() / t_load / 1e9, 2),
        "h2d_frac_of_pcie": round(img.numel() / t_load / 1e9 / PEAK_PCIE_GBPS, 4),
        "overlap_efficiency": round((t_load + t_prefill - t_cold) / min(t_load, t_prefill), 3),
        "decode_ms_per_step": round(dec_ms, 4),
        "decode_tok_s": round(1e3 / dec_ms, 1),
        "decode_hbm_frac": round(dec_bytes / (dec_ms / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
        "decode_roofline": hbm_roofline(dstats, wl.name),
        "kv_export_GBps": round(2 * used / (exp_ms / 1e3) / 1e9, 1),
        "kv_import_GBps": round(2 * used / (imp_ms / 1e3) / 1e9, 1),
        "kv_import_with_readback_GBps": round(2 * used / (statistics.median(imp1) / 1e3) / 1e9, 1),
    }
    st.close()
    img.close()
    return res


def log_decode_breakdown(hs, stages, run, n_steps):
    """Run `run` with every launch of `stages` timed; log the per-kernel
    share of the decode steps."""
    for st in stages:
        hs.hs_stage_read_timing(st.h)
        hs.hs_stage_set_timing_sites(st.h, None)
        hs.hs_stage_set_timing(st.h, 1)
    run()
    agg = {}
    for st in stages:
        hs.hs_stage_set_timing(st.h, 0)
        for k in hs.hs_stage_read_timing(st.h):
            a = agg.setdefault((k["name"], k["site"]), dict(k, launches=0, total_ms=0.0, bytes=0.0))
            a["launches"] += k["launches"]
            a["total_ms"] += k["total_ms"]
            a["bytes"] += k["bytes"]
    tot = sum(a["total_ms"] for a in agg.values())
    steps = n_steps + 2      # run() includes its own two warm-up steps
    log(f"[bench] decode breakdown (every launch timed, {tot / steps:.3f} ms of kernels/step):")
    for a in sorted(agg.values(), key=lambda a: -a["total_ms"])[:10]:
        avg = a["total_ms"] / a["launches"]
        bw = (a["bytes"] / a["launches"]) / (avg / 1e3) / 1e9 if a["bytes"] else 0
        log(f"[bench]   {a['name']:<28} {a['site']:<10} x{a['launches'] // steps:<3} avg "
            f"{avg * 1e3:8.1f} us {100 * a['total_ms'] / tot:5.1f}%  {bw:7.0f} GB/s")
    return list(agg.values())


def hbm_roofline(stats, workload):
    """HBM roofline of the kernel with the most time in `stats` (a decode
    step's launches, every one event-timed): its algorithmic bytes per
    launch over its average duration."""
    dom = max(stats, key=lambda a: a["total_ms"])
    avg_s = dom["total_ms"] / dom["launches"] / 1e3
    per = dom["bytes"] / dom["launches"]
    ach = per / avg_s / 1e9
    return {"bound": "hbm", "kernel": dom["name"], "site": dom["site"],
            "achieved": round(ach, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBPS, 4),
            "traffic": traffic_from_profiles(dom["name"], workload),
            "bytes_per_launch": per, "avg_launch_us": round(avg_s * 1e6, 2)}


def bench_pipeline(wl, args, n_dec=None, oracle_sample=False):
    """A whole pipeline (every stage of the workload) on this GPU, weights
    resident: batched prefill through all stages, then greedy decode steps
    with each step's tokens fed back into the next. Workloads that merge
    decode a few steps in the pipeline, export every stage's KV cache to
    device blobs and import them into a fresh worker holding every layer
    (and once more through pinned host memory), merge the stages into the
    first one (which holds every layer's weights) and decode the n_dec steps
    there. Returns the JSON line as a dict; `value` = prefill tok/s."""
    import numpy as np
    import torch
    from paper_2502_15524_amd import hs, pipeline
    from workloads import gen

    cfg = wl.cfg
    lens = wl.lengths()
    B, T, H, V = len(lens), sum(lens), cfg.hidden, cfg.vocab
    if n_dec is None:
        n_dec = min(wl.decode_steps, args.decode_steps)
    merge = len(wl.stages) > 1 and wl.name.endswith("merge")
    n_pipe = 16 if merge else n_dec          # pipeline steps before a merge
    max_ctx = max(lens) + n_pipe + n_dec + 32
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()
    sp = stream.cuda_stream
    kv_tok_layer = 2 * cfg.n_kv_heads * cfg.head_dim * 2

    # With a merge, the first stage keeps every layer resident (it is the
    # worker the others merge into); it serves only its own range until then.
    t0 = time.perf_counter()
    stages, img_bytes = [], 0
    for k, (b, e) in enumerate(wl.stages):
        rb, re = (0, cfg.n_layers) if merge and k == 0 else (b, e)
        img = pipeline.pinned_image(cfg, rb, re)
        st = pipeline.Stage(cfg, b, e, max_seqs=B + 2, max_ctx=max_ctx, max_batch_tokens=T,
                            resident=(rb, re))
        st.load(img, 64 << 20)
        st.sync()
        img.close()
        img_bytes += hs.hs_weight_layout(pipeline.hs_cfg(cfg), b, e)[1]
        stages.append(st)
    log(f"[bench] {wl.name}: {len(stages)} stage(s) {wl.stages}, {img_bytes / 1e9:.2f} GB of "
        f"serving weights loaded in {time.perf_counter() - t0:.1f} s; batch {B}, {T} prompt "
        f"tokens")

    toks = torch.from_numpy(gen.tokens(V, T, wl.seed)).to(dev)
    hid = [torch.empty((T, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    nxt = torch.empty(B, dtype=torch.int32, device=dev)
    ids_next = [10_000]
    if args.traffic_probe:
        return pipeline_probe(wl, args, stages, toks, hid, nxt, lens, max_ctx, stream)

    def prefill_all():
        ids = list(range(ids_next[0], ids_next[0] + B))
        ids_next[0] += B
        x = toks
        for i, st in enumerate(stages):
            out = nxt if i == len(stages) - 1 else hid[i % 2]
            st.prefill(ids, lens, x.data_ptr(), out.data_ptr(), 0, sp)
            x = out
        return ids

    def free(ids):
        for st in stages:
            for i in ids:
                hs.hs_seq_free(st.h, i)

    def timed(fn, reps):
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        t0 = time.perf_counter()
        out = [fn() for _ in range(reps)]
        ev1.record(stream)
        stream.synchronize()
        return max(ev0.elapsed_time(ev1), (time.perf_counter() - t0) * 1e3) / reps, out

    # prefill: one untimed step (first launches load their kernels), one
    # with every launch timed (breakdown), then timed steps
    free(prefill_all())
    stream.synchronize()
    for st in stages:
        hs.hs_stage_read_timing(st.h)
        hs.hs_stage_set_timing(st.h, 1)
    free(prefill_all())
    stream.synchronize()
    stats = {}
    for st in stages:
        hs.hs_stage_set_timing(st.h, 0)
        for k in hs.hs_stage_read_timing(st.h):
            key = (k["name"], k["site"])
            a = stats.setdefault(key, dict(k, launches=0, total_ms=0.0, flops=0.0))
            a["launches"] += k["launches"]
            a["total_ms"] += k["total_ms"]
            a["flops"] += k["flops"]
    kern_ms = sum(a["total_ms"] for a in stats.values())
    flops_step = sum(a["flops"] for a in stats.values())
    for a in sorted(stats.values(), key=lambda a: -a["total_ms"])[:8]:
        avg = a["total_ms"] / a["launches"]
        rate = (a["flops"] / a["launches"]) / (avg / 1e3) / 1e12 if a["flops"] else 0
        log(f"[bench]   {a['name']:<28} {a['site']:<10} x{a['launches']:<4} avg "
            f"{avg * 1e3:9.1f} us {100 * a['total_ms'] / kern_ms:5.1f}%  {rate:7.1f} TFLOP/s")
    dom = max(stats.values(), key=lambda a: a["total_ms"])
    reps = max(1, min(args.steps, 5))
    for st in stages:
        hs.hs_stage_set_timing_sites(st.h, dom["site"])
        hs.hs_stage_set_timing(st.h, 1)
    ms_pre, _ = timed(lambda: free(prefill_all()), reps)
    timed_stats = []
    for st in stages:
        hs.hs_stage_set_timing(st.h, 0)
        hs.hs_stage_set_timing_sites(st.h, None)
        timed_stats += [k for k in hs.hs_stage_read_timing(st.h)
                        if k["name"] == dom["name"] and k["site"] == dom["site"]]
    d_launch = sum(k["launches"] for k in timed_stats)
    d_avg_s = sum(k["total_ms"] for k in timed_stats) / d_launch / 1e3
    d_flops = sum(k["flops"] for k in timed_stats) / d_launch
    achieved = d_flops / d_avg_s / 1e12
    log(f"[bench] prefill {ms_pre:.2f} ms = {T / ms_pre * 1e3:,.0f} tok/s "
        f"({flops_step / (ms_pre / 1e3) / 1e12:.0f} TFLOP/s, "
        f"{flops_step / (ms_pre / 1e3) / 1e12 / PEAK_BF16_TFLOPS:.1%} of MFMA peak); dominant "
        f"{dom['name']} ({dom['site']}) {d_avg_s * 1e6:.1f} us, {achieved:.0f} TFLOP/s")

    # greedy decode: the last stage's tokens are the next step's input
    tokb = [torch.empty(B, dtype=torch.int32, device=dev) for _ in range(2)]
    hbuf = [torch.empty((B, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    cur = [0]

    def one_step(sts, ids):
        xi = tokb[cur[0]]
        for i, st in enumerate(sts):
            out = tokb[cur[0] ^ 1] if i == len(sts) - 1 else hbuf[i % 2]
            st.decode(ids, xi.data_ptr(), out.data_ptr(), 0, sp)
            xi = out
        cur[0] ^= 1

    def decode_steps(sts, ids, n):
        ms, _ = timed(lambda: one_step(sts, ids), n)
        return ms

    ids = prefill_all()
    tokb[0].copy_(nxt)
    cur[0] = 0
    ctx0 = np.array(lens, np.float64)          # cached tokens before the next step
    for _ in range(2):
        one_step(stages, ids)
    ctx0 += 2
    ms_dec = decode_steps(stages, ids, n_pipe)
    kv_read = (float((ctx0 + (n_pipe + 1) / 2.0).sum()) * kv_tok_layer * cfg.n_layers)
    ctx0 += n_pipe
    dstats = log_decode_breakdown(hs, stages, lambda: [one_step(stages, ids) for _ in range(4)], 2)
    ctx0 += 4
    w_bytes = img_bytes - (V * H * 2) + B * H * 2   # embedding: B rows per step
    dec_bytes = w_bytes + kv_read + B * kv_tok_layer * cfg.n_layers
    log(f"[bench] decode B={B} {ms_dec:.3f} ms/step = {B / ms_dec * 1e3:,.0f} tok/s, "
        f"{dec_bytes / (ms_dec / 1e3) / 1e9:,.0f} GB/s "
        f"({dec_bytes / (ms_dec / 1e3) / 1e9 / PEAK_HBM_GBPS:.1%} of HBM; weights "
        f"{w_bytes / 1e9:.2f} GB + KV {kv_read / 1e9:.2f} GB per step, {n_pipe} greedy steps)")
    res_extra = {}
    if merge:
        # KV export of every stage to device blobs, and import of all of them
        # into a fresh worker holding every layer's pools
        blobs, heads, exp_ms, moved = [], [], [], 0
        for st in stages:
            size = hs.hs_kv_export_size(st.h, ids)
            blob = torch.empty(size, dtype=torch.uint8, device=dev)
            hs.hs_kv_export(st.h, ids, blob.data_ptr(), size, sp)   # warm
            ms, _ = timed(lambda: hs.hs_kv_export(st.h, ids, blob.data_ptr(), size, sp), 5)
            exp_ms.append(ms)
            blobs.append((blob, size))
            heads.append(hs.hs_kv_export_head(st.h, ids))
            moved += size - len(heads[-1])
        tgt = pipeline.Stage(cfg, 0, cfg.n_layers, max_seqs=B + 2, max_ctx=max_ctx,
                             max_batch_tokens=T)
        many = [(b.data_ptr(), n, hd) for (b, n), hd in zip(blobs, heads)]
        hs.hs_kv_import_many(tgt.h, many, sp)        # warm: sizes the copy descriptors
        imp_ms, imp1_ms = [], []
        for r in range(6):
            for i in ids:
                hs.hs_seq_free(tgt.h, i)
            if r % 2:        # one hs_kv_import per blob (each reads its header back)
                ms_r, _ = timed(lambda: [hs.hs_kv_import(tgt.h, b.data_ptr(), n, sp)
                                         for b, n in blobs], 1)
                imp1_ms.append(ms_r)
            else:            # all blobs in one call, headers from the exporters
                ms_r, _ = timed(lambda: hs.hs_kv_import_many(tgt.h, many, sp), 1)
                imp_ms.append(ms_r)
        # host-staged form: each stage's blob leaves the GPU in 64 MiB chunks
        # into pinned host memory, and the target loads them back chunk by
        # chunk (the cross-machine path; bounded by the host link)
        hosts = [pipeline.PinnedBuffer(n) for _, n in blobs]
        for r in range(2):      # the first round sizes the staging buffers
            t = time.perf_counter()
            for st, hb, (_, n) in zip(stages, hosts, blobs):
                hs.hs_kv_export_host(st.h, ids, hb.data_ptr(), n, 64 << 20, sp)
            for st in stages:
                st.sync()
            ms_exp_host = (time.perf_counter() - t) * 1e3
        for r in range(2):
            for i in ids:
                hs.hs_seq_free(tgt.h, i)
            torch.cuda.synchronize()
            t = time.perf_counter()
            for hb, (_, n) in zip(hosts, blobs):
                hs.hs_kv_import_host(tgt.h, hb.data_ptr(), n, 64 << 20, sp)
            tgt.sync()
            stream.synchronize()
            ms_imp_host = (time.perf_counter() - t) * 1e3
        for hb in hosts:
            hb.close()
        log(f"[bench] host-staged KV migration: export to host {ms_exp_host:.2f} ms "
            f"({moved / (ms_exp_host / 1e3) / 1e9:.1f} GB/s over the host link), import from "
            f"host {ms_imp_host:.2f} ms ({moved / (ms_imp_host / 1e3) / 1e9:.1f} GB/s)")
        tgt.close()
        ms_imp = statistics.median(imp_ms)
        ms_exp = sum(exp_ms)
        # reference: a plain device-to-device copy of the same bytes
        copy_ms = 0.0
        with torch.cuda.stream(stream):
            for b, n in blobs:
                dst_b = torch.empty_like(b)
                dst_b.copy_(b)
                ms_c, _ = timed(lambda: dst_b.copy_(b), 5)
                copy_ms += ms_c
                del dst_b
        del blobs
        ms_imp1 = statistics.median(imp1_ms)
        log(f"[bench] KV export {moved / 1e9:.2f} GB in {ms_exp:.2f} ms "
            f"({2 * moved / (ms_exp / 1e3) / 1e9:,.0f} GB/s), import {ms_imp:.2f} ms "
            f"({2 * moved / (ms_imp / 1e3) / 1e9:,.0f} GB/s; blob by blob with header "
            f"read-backs {ms_imp1:.2f} ms); a plain device copy of the "
            f"same blobs {copy_ms:.2f} ms ({2 * moved / (copy_ms / 1e3) / 1e9:,.0f} GB/s)")
        # the merge itself: stage 0 takes over every layer (drain, block
        # copies into its pools, serving range extended), then decodes alone
        ms_merge, _ = timed(lambda: hs.hs_stage_merge(stages[0].h, [st.h for st in stages[1:]],
                                                      sp), 1)
        ms_dec_m = decode_steps([stages[0]], ids, n_dec)
        kv_m = float((ctx0 + (n_dec + 1) / 2.0).sum()) * kv_tok_layer * cfg.n_layers
        dec_bytes_m = w_bytes + kv_m + B * kv_tok_layer * cfg.n_layers
        mstats = log_decode_breakdown(hs, [stages[0]],
                                      lambda: [one_step([stages[0]], ids) for _ in range(4)], 2)
        log(f"[bench] merge {ms_merge:.2f} ms; merged-worker decode B={B} {ms_dec_m:.3f} "
            f"ms/step = {B / ms_dec_m * 1e3:,.0f} tok/s over {n_dec} greedy steps "
            f"({dec_bytes_m / (ms_dec_m / 1e3) / 1e9 / PEAK_HBM_GBPS:.1%} of HBM)")

        def kv_roof(ms):
            ach = 2 * moved / (ms / 1e3) / 1e9
            return {"bound": "hbm", "kernel": "kv_copy", "achieved": round(ach, 1),
                    "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBPS, 4),
                    "traffic": traffic_from_profiles("kv_copy", wl.name),
                    "bytes_per_op": 2 * moved,
                    "device_copy_ceiling_GBps": round(2 * moved / (copy_ms / 1e3) / 1e9, 1)}
        res_extra = {"kv_export_ms": round(ms_exp, 3), "kv_import_ms": round(ms_imp, 3),
                     "kv_import_blob_by_blob_ms": round(ms_imp1, 3),
                     "device_copy_same_bytes_ms": round(copy_ms, 3),
                     "kv_bytes": moved,
                     "kv_export_GBps": round(2 * moved / (ms_exp / 1e3) / 1e9, 1),
                     "kv_import_GBps": round(2 * moved / (ms_imp / 1e3) / 1e9, 1),
                     "kv_export_roofline": kv_roof(ms_exp),
                     "kv_import_roofline": kv_roof(ms_imp),
                     "merge_ms": round(ms_merge, 3),
                     "kv_export_host_ms": round(ms_exp_host, 3),
                     "kv_export_host_GBps": round(moved / (ms_exp_host / 1e3) / 1e9, 2),
                     "kv_import_host_ms": round(ms_imp_host, 3),
                     "kv_import_host_GBps": round(moved / (ms_imp_host / 1e3) / 1e9, 2),
                     "merged_decode_steps": n_dec,
                     "merged_decode_ms_per_step": round(ms_dec_m, 4),
                     "merged_decode_tok_s": round(B / ms_dec_m * 1e3, 1),
                     "merged_decode_hbm_frac": round(dec_bytes_m / (ms_dec_m / 1e3) / 1e9 /
                                                     PEAK_HBM_GBPS, 4),
                     "merged_decode_roofline": hbm_roofline(mstats, wl.name)}
    res = {
        "metric": METRIC, "value": round(T / ms_pre * 1e3, 1), "unit": "tok/s", "n_gpus": 1,
        "steps": reps, "warmup": 1, "ms_per_step": round(ms_pre, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "model_shape": cfg.name, "stages": wl.stages,
                   "batch": B, "prompt_tokens": T, "decode_steps": n_dec},
        "roofline": {"bound": "mfma", "kernel": dom["name"], "achieved": round(achieved, 1),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic_from_profiles(dom["name"], wl.name),
                     "flops_per_launch": d_flops, "avg_launch_us": round(d_avg_s * 1e6, 2)},
        "cpu_baseline": None,
        "prefill_ms": round(ms_pre, 3),
        "prefill_mfma_frac_step": round(flops_step / (ms_pre / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "decode_steps_timed": n_pipe, "decode_fed_back": "greedy tokens of the previous step",
        "decode_ms_per_step": round(ms_dec, 4), "decode_tok_s": round(B / ms_dec * 1e3, 1),
        "decode_hbm_frac": round(dec_bytes / (ms_dec / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
        "decode_roofline": hbm_roofline(dstats, wl.name),
    }
    res.update(res_extra)
    for st in stages:
        st.close()
    if oracle_sample:
        res["cpu_baseline"] = oracle_sample_pipeline(wl, T, B, lens, moved if merge else 0)
    return res


def traffic_calibration_copies(torch, dev):
    """Two device copies of 256 MiB: the known-size dispatches that scale
    the FETCH_SIZE / WRITE_SIZE counters of a probe run."""
    src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    dstc = torch.empty_like(src)
    src.fill_(1)
    for _ in range(2):
        dstc.copy_(src)
    torch.cuda.synchronize()


def pipeline_probe(wl, args, stages, toks, hid, nxt, lens, max_ctx, stream):
    """Workload for hardware-counter passes of a whole pipeline: one prefill,
    4 decode steps, and for a merge workload one export per stage and one
    import of all blobs; then the calibration copies."""
    import torch
    from paper_2502_15524_amd import hs, pipeline
    cfg = wl.cfg
    B, T, H = len(lens), sum(lens), cfg.hidden
    sp = stream.cuda_stream
    ids = list(range(B))
    x = toks
    for i, st in enumerate(stages):
        out = nxt if i == len(stages) - 1 else hid[i % 2]
        st.prefill(ids, lens, x.data_ptr(), out.data_ptr(), 0, sp)
        x = out
    tok = [nxt.clone(), torch.empty_like(nxt)]
    hb = [torch.empty((B, H), dtype=torch.bfloat16, device=nxt.device) for _ in range(2)]
    for k in range(4):
        x = tok[k % 2]
        for i, st in enumerate(stages):
            out = tok[(k + 1) % 2] if i == len(stages) - 1 else hb[i % 2]
            st.decode(ids, x.data_ptr(), out.data_ptr(), 0, sp)
            x = out
    what = "1 prefill, 4 decode steps"
    if wl.name.endswith("merge"):
        many = []
        for st in stages:
            n = hs.hs_kv_export_size(st.h, ids)
            blob = torch.empty(n, dtype=torch.uint8, device=nxt.device)
            hs.hs_kv_export(st.h, ids, blob.data_ptr(), n, sp)
            many.append((blob, n, hs.hs_kv_export_head(st.h, ids)))
        tgt = pipeline.Stage(cfg, 0, cfg.n_layers, max_seqs=B + 2, max_ctx=max_ctx,
                             max_batch_tokens=T)
        hs.hs_kv_import_many(tgt.h, [(b.data_ptr(), n, hd) for b, n, hd in many], sp)
        stream.synchronize()
        tgt.close()
        what += f", {len(stages)} KV exports and one import of all of them"
    stream.synchronize()
    for st in stages:
        st.close()
    traffic_calibration_copies(torch, nxt.device)
    log(f"[bench] traffic probe done ({wl.name}): {what}, 2 copies of 268435456 bytes")
    return None


_EPI_NAMES = ["store", "resid", "swiglu", "f32", "qkv_rope"]


def bench_kernel_name(rocprof_name):
    """The launch name bench.py reports (LaunchInfo) for a rocprofv3 kernel
    name, and the source file of the kernel; (None, None) for others."""
    import re
    m = re.search(r"gemm_ring<(\d+), (\d+), \d+, \d+, (true|false), (\d+)[,>]", rocprof_name)
    if m:
        sk = "sk" if m.group(3) == "true" else ""
        return f"gemm_r{m.group(1)}x{m.group(2)}{sk}_{_EPI_NAMES[int(m.group(4))]}", "k_gemm"
    m = re.search(r"gemm_skinny<\d+, \d+, \d+, (\d+), (true|false), \d+[,>]", rocprof_name)
    if m:
        norm = "norm_" if m.group(2) == "true" else ""
        return f"gemm_skinny_{norm}{_EPI_NAMES[int(m.group(1))]}", "k_gemm"
    m = re.search(r"attn_prefill_kernel<(\d+),", rocprof_name)
    if m:
        return f"attn_prefill_d{m.group(1)}", "k_attn"
    if "attn_decode" in rocprof_name:
        return "attn_decode", "k_attn"
    for k in ("kv_copy", "rmsnorm", "embed", "argmax", "rope_kv"):
        if k + "_kernel" in rocprof_name or (k == "argmax" and "argmax" in rocprof_name):
            return k, "k_misc"
    return None, None


def summarize_counters(fetch_csv, write_csv, workload):
    """Per-kernel HBM traffic of a probe run from two rocprofv3 counter
    passes (FETCH_SIZE, WRITE_SIZE; KiB per dispatch), each scaled by what it
    reads for the two 256 MiB calibration copies at the end of the run.
    Prints a markdown table and the machine-readable "traffic:" lines that
    traffic_from_profiles() reads."""
    import csv
    from collections import defaultdict

    def load(path):
        rows = list(csv.DictReader(open(path)))
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        return rows
    f_rows, w_rows = load(fetch_csv), load(write_csv)
    copy_f = [float(r["Counter_Value"]) for r in f_rows if "copy" in r["Kernel_Name"].lower()][-2:]
    copy_w = [float(r["Counter_Value"]) for r in w_rows if "copy" in r["Kernel_Name"].lower()][-2:]
    kib = 268435456 / 1024
    sf, sw = kib / (sum(copy_f) / 2), kib / (sum(copy_w) / 2)
    per = defaultdict(lambda: [0, 0.0, 0.0])
    for rows, idx in ((f_rows, 1), (w_rows, 2)):
        for r in rows:
            per[r["Kernel_Name"]][idx] += float(r["Counter_Value"])
            if idx == 1:
                per[r["Kernel_Name"]][0] += 1
    csrc = os.path.join(ROOT, "paper_2502_15524_amd", "csrc")
    print(f"calibration: FETCH_SIZE x{sf:.3f}, WRITE_SIZE x{sw:.3f} (two copies of 268435456 B)")
    print("| kernel (rocprofv3 name) | bench name | dispatches | FETCH_SIZE KiB / dispatch | "
          "WRITE_SIZE KiB / dispatch | calibrated HBM bytes / dispatch |")
    print("|---|---|---|---|---|---|")
    lines, attn = [], 0.0
    owners = defaultdict(set)        # bench name -> rocprofv3 kernels behind it
    for name in per:
        owners[bench_kernel_name(name)[0]].add(name)
    for name, (n, f, w) in sorted(per.items(), key=lambda kv: -(kv[1][1] + kv[1][2])):
        bname, src = bench_kernel_name(name)
        if not bname or n == 0:
            continue
        fb, wb = f / n, w / n
        hbm = (fb * sf + wb * sw) * 1024
        short = name.split("(")[0].replace("void ", "")
        print(f"| `{short}` | {bname} | {n} | {fb:,.1f} | {wb:,.1f} | {hbm:,.0f} |")
        if bname == "attn_decode":
            attn += hbm   # split + combine kernels form one call
            src_attn = src
            continue
        if bname == "kv_copy" and workload.endswith("merge"):
            # the probe's copies are one export of every stage and one import
            # of all blobs: two operations of equal size
            hbm = (f * sf + w * sw) * 1024 / 2
        elif len(owners[bname]) > 1 or bname.endswith("_resid"):
            continue      # the o and down launch sites share the name: no line
        lines.append(f"traffic: kernel={bname} workload={workload} hbm_bytes_per_launch="
                     f"{int(hbm)} {src}_sha256={_sha(os.path.join(csrc, src + '.hip'))}")
    if attn:
        lines.append(f"traffic: kernel=attn_decode workload={workload} hbm_bytes_per_launch="
                     f"{int(attn)} {src_attn}_sha256={_sha(os.path.join(csrc, src_attn + '.hip'))}")
    print()
    for l in lines:
        print(l)


def oracle_sample_pipeline(wl, T, B, lens, kv_bytes):
    """The oracle on a bounded sample of the same workload: the prefill of
    the whole batch through one layer (scaled to all layers) and 8 decode
    steps of the batch through that layer (scaled); for a merge workload also
    the oracle's blob codec packing one layer's cache of every sequence
    (GB/s)."""
    import numpy as np
    from oracle import kvblob
    from oracle.llama import Stage
    from workloads import gen
    cfg = wl.cfg
    L = cfg.n_layers
    W = layer_weights(cfg, [1])
    st = Stage(cfg, W, 1, 2)
    x = gen.hidden_input(T, cfg.hidden, wl.seed)

    def pre(i):
        st.prefill(list(range(100 * i, 100 * i + B)), lens, x)
        if i == 0:
            return
        for sid in range(100 * i, 100 * i + B):
            st.drop(sid)
    reps, dt = oracle_timed(pre, 3.0)
    ids = list(range(B))          # cache of prefill 0 kept for decode
    xd = gen.hidden_input(B, cfg.hidden, wl.seed + 1)
    t0 = time.perf_counter()
    for _ in range(8):
        st.decode(ids, xd)
    dec_s = (time.perf_counter() - t0) / 8
    hi = host_info()
    res = {"value": round(T / (dt / reps * L), 2), "unit": "tok/s", "cores": hi["blas_threads"],
           "kind": "oracle",
           "sample": f"{reps} prefills of the batch ({T} tokens) through one decoder layer "
                     f"({dt:.1f} s), scaled to {L} layers (head not included)",
           "decode_ms_per_step": round(dec_s * 1e3 * L, 1),
           "decode_sample": f"8 decode steps of the batch through the same layer "
                            f"({dec_s * 8:.2f} s), scaled to {L} layers"}
    if kv_bytes:
        K = np.zeros((1, max(lens), cfg.n_kv_heads, cfg.head_dim), np.uint16)
        seqs = [(i, K[:, :n], K[:, :n]) for i, n in enumerate(lens)]
        t0 = time.perf_counter()
        blob = kvblob.pack(0, 1, cfg.n_kv_heads, cfg.head_dim, 16, seqs)
        pk = time.perf_counter() - t0
        res["kv_pack_GBps"] = round(len(blob) / pk / 1e9, 3)
        res["kv_pack_sample"] = (f"oracle blob codec packing one layer of all {B} sequences "
                                 f"({len(blob) / 1e6:.1f} MB in {pk:.2f} s)")
    res.update(hi)
    return res


def bench_cold_stage(wl, args):
    """Cold TTFT of the workload's first stage: its weights streamed from
    pinned host memory in 64 MiB chunks while it prefills the whole batch
    (each layer starts when its bytes land); host wall clock from the first
    chunk enqueue to the stage's output being ready, median of 5; the load
    alone; the warm prefill; and the cold TTFT including the stage's
    creation (median of 3)."""
    import torch
    from paper_2502_15524_amd import hs, pipeline
    from workloads import gen

    cfg = wl.cfg
    lens = wl.lengths()
    B, T, H = len(lens), sum(lens), cfg.hidden
    b, e = wl.stages[0]
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()
    sp = stream.cuda_stream
    t = time.perf_counter()
    img = pipeline.pinned_image(cfg, b, e)
    W = img.numel()
    log(f"[bench] {wl.name} stage [{b}, {e}): image {W / 1e9:.2f} GB packed in "
        f"{time.perf_counter() - t:.1f} s")
    toks = torch.from_numpy(gen.tokens(cfg.vocab, T, wl.seed)).to(dev)
    out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
    kw = dict(max_seqs=B + 1, max_ctx=max(lens) + 8, max_batch_tokens=T)
    st = pipeline.Stage(cfg, b, e, **kw)
    chunk = args.cold_chunk_mb << 20
    ids = list(range(B))

    def prefill(s):
        s.prefill(ids, lens, toks.data_ptr(), out.data_ptr(), 0, sp)

    def free(s):
        for i in ids:
            hs.hs_seq_free(s.h, i)
    cold, load_only, warm, submit = [], [], [], []
    for r in range(6):
        hs.hs_stage_invalidate_weights(st.h)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st.load(img, chunk)
        submit.append(time.perf_counter() - t0)
        prefill(st)
        stream.synchronize()
        dt = time.perf_counter() - t0
        st.sync()
        free(st)
        if r:
            cold.append(dt)
        hs.hs_stage_invalidate_weights(st.h)
        t0 = time.perf_counter()
        st.load(img, chunk)
        st.sync()
        if r:
            load_only.append(time.perf_counter() - t0)
        t0 = time.perf_counter()
        prefill(st)
        stream.synchronize()
        if r:
            warm.append(time.perf_counter() - t0)
        free(st)
    with_create = []
    for r in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        s2 = pipeline.Stage(cfg, b, e, **kw)
        s2.load(img, chunk)
        prefill(s2)
        stream.synchronize()
        with_create.append(time.perf_counter() - t0)
        s2.close()
    st.close()
    img.close()
    t_cold, t_load = statistics.median(cold), statistics.median(load_only)
    t_warm = statistics.median(warm)
    log(f"[bench] {wl.name} stage 0 cold TTFT {t_cold * 1e3:.1f} ms (load only "
        f"{t_load * 1e3:.1f} ms = {W / t_load / 1e9:.1f} GB/s, warm prefill {t_warm * 1e3:.1f} "
        f"ms, with creation {statistics.median(with_create) * 1e3:.1f} ms; submitting the "
        f"{-(-W // chunk)} chunks took {statistics.median(submit[1:]) * 1e3:.1f} ms of host time)")
    ach = W / t_cold / 1e9
    return {
        "metric": "cold TTFT (weights in host) ms", "value": round(t_cold * 1e3, 2),
        "unit": "ms", "higher_is_better": False,
        "config": {"workload": wl.name, "model_shape": cfg.name, "stage": [b, e],
                   "batch": B, "prompt_tokens": T},
        "cold_ttft_ms": round(t_cold * 1e3, 2),
        "cold_ttft_with_create_ms": round(statistics.median(with_create) * 1e3, 2),
        "load_only_ms": round(t_load * 1e3, 2),
        "warm_prefill_ms": round(t_warm * 1e3, 2),
        "image_bytes": W, "chunk_bytes": chunk,
        "chunk_submit_ms": round(statistics.median(submit[1:]) * 1e3, 2),
        "overlap_efficiency": round((t_load + t_warm - t_cold) / min(t_load, t_warm), 3),
        "roofline": {"bound": "host_link", "kernel": "weight upload (hipMemcpyAsync)",
                     "achieved": round(ach, 2), "peak": PEAK_PCIE_GBPS, "unit": "GB/s",
                     "frac": round(ach / PEAK_PCIE_GBPS, 4), "traffic": None,
                     "note": "image bytes over the cold TTFT (upload and prefill overlapped)"},
        "cpu_baseline": None,
        "cpu_baseline_note": "a cold start is a host-to-GPU transfer; the oracle has none",
    }


def bench_scale_down(wl, args):
    """Scaling down: stage 0 serves layers [0, L/4) but reserves memory for
    all L; after the batch's prefill it loads the remaining layers in the
    background while the 4-stage pipeline keeps decoding, and once they have
    landed it absorbs the other stages' KV cache (hs_stage_merge) and decodes
    alone. Per-token (per-step) times are recorded, and a pipeline-only run
    of the same length is the reference."""
    import numpy as np
    import torch
    from paper_2502_15524_amd import hs, pipeline
    from workloads import gen

    cfg = wl.cfg
    L = cfg.n_layers
    lens = wl.lengths()
    B, T, H, V = len(lens), sum(lens), cfg.hidden, cfg.vocab
    n_dec = wl.decode_steps
    max_ctx = max(lens) + n_dec + 16
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()
    sp = stream.cuda_stream
    c = pipeline.hs_cfg(cfg)

    t0 = time.perf_counter()
    full = pipeline.pinned_image(cfg, 0, L)
    descs, nbytes = hs.hs_weight_layout(c, 0, L)
    b0, e0 = wl.stages[0]
    # stage 0's own part: the embedding and its layers (the final norm and the
    # head, layer -1 like the embedding, sit at the end of the image)
    first_end = max(d["offset"] + d["bytes"] for d in descs
                    if 0 <= d["layer"] < e0 or d["kind"] == hs.HS_W_EMBED)
    chunk = 64 << 20
    s0 = pipeline.Stage(cfg, b0, e0, max_seqs=B + 2, max_ctx=max_ctx, max_batch_tokens=T,
                        resident=(0, L))
    for off in range(0, first_end, chunk):
        hs.hs_stage_load_chunk(s0.h, off, full.data_ptr() + off, min(chunk, first_end - off))
    s0.sync()
    stages = [s0]
    for b, e in wl.stages[1:]:
        img = pipeline.pinned_image(cfg, b, e)
        st = pipeline.Stage(cfg, b, e, max_seqs=B + 2, max_ctx=max_ctx, max_batch_tokens=T)
        st.load(img, chunk)
        st.sync()
        img.close()
        stages.append(st)
    log(f"[bench] {wl.name}: stages {wl.stages}; stage 0 resident [0, {L}) with "
        f"{first_end / 1e9:.2f} of {nbytes / 1e9:.2f} GB loaded; set-up "
        f"{time.perf_counter() - t0:.1f} s")

    toks = torch.from_numpy(gen.tokens(V, T, wl.seed)).to(dev)
    hid = [torch.empty((T, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    hb = [torch.empty((B, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    nxt = torch.empty(B, dtype=torch.int32, device=dev)

    def prefill(sts, ids):
        x = toks
        for i, st in enumerate(sts):
            out = nxt if i == len(sts) - 1 else hid[i % 2]
            st.prefill(ids, lens, x.data_ptr(), out.data_ptr(), 0, sp)
            x = out
        stream.synchronize()

    def step(sts, ids):
        x = nxt.clone()
        t = time.perf_counter()
        for i, st in enumerate(sts):
            out = nxt if i == len(sts) - 1 else hb[i % 2]
            st.decode(ids, x.data_ptr(), out.data_ptr(), 0, sp)
            x = out
        stream.synchronize()
        return (time.perf_counter() - t) * 1e3

    # reference: the pipeline decodes all tokens (no consolidation)
    ids = list(range(100, 100 + B))
    prefill(stages, ids)
    ref = [step(stages, ids) for _ in range(n_dec)]
    for st in stages:
        for i in ids:
            hs.hs_seq_free(st.h, i)
    log(f"[bench] pipeline only: {np.mean(ref):.3f} ms/token-step "
        f"({sum(ref):.1f} ms for {n_dec} steps)")

    # scale-down run
    ids = list(range(200, 200 + B))
    prefill(stages, ids)
    t_load0 = time.perf_counter()
    for off in range(first_end, nbytes, chunk):
        hs.hs_stage_load_chunk(s0.h, off, full.data_ptr() + off, min(chunk, nbytes - off))
    times, merged_at, t_loaded, ms_merge = [], None, None, None
    cur = stages
    for k in range(n_dec):
        times.append(step(cur, ids))
        if merged_at is None:
            _, wm = hs.hs_stage_loaded(s0.h)
            if wm == nbytes:
                t_loaded = (time.perf_counter() - t_load0) * 1e3
                t = time.perf_counter()
                hs.hs_stage_merge(s0.h, [st.h for st in stages[1:]], sp)
                stream.synchronize()
                ms_merge = (time.perf_counter() - t) * 1e3
                merged_at = k + 1
                cur = [s0]
    assert merged_at is not None, "background load did not finish within the decode steps"
    during = times[:merged_at]
    after = times[merged_at:]
    total_sd = sum(times) + ms_merge
    log(f"[bench] scale-down: background load of {(nbytes - first_end) / 1e9:.2f} GB landed "
        f"after {t_loaded:.1f} ms ({(nbytes - first_end) / (t_loaded / 1e3) / 1e9:.1f} GB/s); "
        f"{merged_at} steps during the load at {np.mean(during):.3f} ms/step "
        f"(pipeline only {np.mean(ref):.3f}); merge {ms_merge:.2f} ms; "
        f"{len(after)} steps after at {np.mean(after) if after else float('nan'):.3f} ms/step; "
        f"generation {total_sd:.1f} ms vs {sum(ref):.1f} ms pipeline only")
    res = {
        "metric": METRIC, "value": round(B * n_dec / (total_sd / 1e3), 1), "unit": "tok/s",
        "n_gpus": 1, "steps": n_dec, "warmup": 0, "ms_per_step": round(total_sd / n_dec, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "model_shape": cfg.name, "stages": wl.stages,
                   "batch": B, "prompt_len": lens[0], "generated_tokens": n_dec},
        "roofline": None, "cpu_baseline": None,
        "background_load_bytes": nbytes - first_end,
        "background_load_ms": round(t_loaded, 2),
        "background_load_GBps": round((nbytes - first_end) / (t_loaded / 1e3) / 1e9, 2),
        "steps_during_load": merged_at,
        "ms_per_step_during_load": round(float(np.mean(during)), 4),
        "ms_per_step_pipeline_only": round(float(np.mean(ref)), 4),
        "merge_ms": round(ms_merge, 3),
        "ms_per_step_after_merge": round(float(np.mean(after)), 4) if after else None,
        "generation_ms_scale_down": round(total_sd, 2),
        "generation_ms_pipeline_only": round(sum(ref), 2),
        "per_step_ms_scale_down": [round(t, 3) for t in times],
        "per_step_ms_pipeline_only": [round(t, 3) for t in ref],
    }
    for st in stages:
        st.close()
    full.close()
    return res


if __name__ == "__main__":
    main()
