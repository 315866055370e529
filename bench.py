"""Benchmark of the pipeline-stage engine on one MI355X.

Default workload: the Llama-2-7B-shaped model cut into 4 stages; the second
stage (layers 8-15) serves one 512-token prompt (batch 1). One step is one
prefill of that prompt through the stage with its weights resident in HBM
(the stage's contribution to TTFT); `value` is prompt tokens per second over
the K timed steps. Reported beside it:
  * cold TTFT: weights streamed from pinned host memory in chunks while the
    stage prefills (each layer starts when its bytes land), host wall clock
    from the first chunk enqueue to the output being ready (PCIe-inclusive);
  * decode: batch-1 decode steps of the same stage (HBM-bound);
  * KV export / import of the stage's cache (device to device);
  * roofline of the dominant kernel, timed with HIP events on the launch
    stream inside the timed region;
  * the CPU oracle timed on this host on the same prefill.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cold-runs", type=int, default=5)
    ap.add_argument("--decode-steps", type=int, default=64)
    ap.add_argument("--chunk-mb", type=int, default=64)
    ap.add_argument("--copy-streams", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="only run a few warm prefill steps and a 256 MiB device copy "
                         "(the workload for hardware-counter passes)")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def traffic_from_profiles(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summaries
    (profiles/*traffic*.md, a line "traffic: kernel=K hbm_bytes_per_launch=B
    k_gemm_sha256=H"), if they were taken on the current GEMM source; else
    None."""
    import glob
    src = os.path.join(ROOT, "paper_2502_15524_amd", "csrc", "k_gemm.hip")
    with open(src, "rb") as f:
        h = hashlib.sha256(f.read()).hexdigest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*traffic*.md"))):
        with open(path) as f:
            for line in f:
                if not line.startswith("traffic:"):
                    continue
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                if kv.get("kernel") == kernel and kv.get("k_gemm_sha256") == h:
                    return int(kv["hbm_bytes_per_launch"])
    return None


def cpu_baseline(wl, x_f32, stage_range, min_seconds=12.0):
    """The oracle, as it stands, on the same prefill (all 512 tokens, all 8
    layers of the stage), on this host's cores."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle.llama import Stage, SyntheticWeights
    cfg = wl.cfg
    W = SyntheticWeights(cfg)
    b, e = stage_range
    for l in range(b, e):               # draw the weights before timing
        for k in ("wq", "wk", "wv", "wo", "wgate", "wup", "wdown"):
            W(l, k)
    st = Stage(cfg, W, b, e)
    reps, dt = 0, 0.0
    while dt < min_seconds:            # repeat the prefill for a bounded sample
        t0 = time.perf_counter()
        st.prefill([reps], [x_f32.shape[0]], x_f32)
        dt += time.perf_counter() - t0
        st.drop(reps)
        reps += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()
                   if p.get("user_api") == "blas"] or [1])
    return {"value": round(reps * x_f32.shape[0] / dt, 2), "unit": "tok/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"{reps} full prefills of the {x_f32.shape[0]}-token prompt through "
                      f"layers {b}-{e - 1} (numpy float32, {dt:.1f} s in total)",
            "host_cpus": os.cpu_count()}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the stage engine "
              "has no multi-GPU path in this build", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2502_15524_amd import hs, pipeline
    from workloads import WORKLOADS, gen

    wl = WORKLOADS["7b-stage8-15-cold"]
    cfg = wl.cfg
    b, e = wl.stages[wl.bench_stage]
    P = wl.prompt_lens[0]
    H = cfg.hidden
    assert torch.cuda.is_available()
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream()
    sp = stream.cuda_stream

    t = time.perf_counter()
    img = pipeline.pinned_image(cfg, b, e)
    log(f"[bench] packed stage image {img.numel() / 1e9:.3f} GB in {time.perf_counter() - t:.1f} s")
    x_f32 = gen.hidden_input(P, H, wl.seed)
    x = torch.from_numpy(gen.to_bf16_bits(x_f32).view(np.int16)).view(torch.bfloat16).to(dev)
    out = torch.empty((P, H), dtype=torch.bfloat16, device=dev)
    max_ctx = P + args.decode_steps + 16
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
        stream.synchronize()
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        dstc = torch.empty_like(src)
        src.fill_(1)
        for _ in range(2):
            dstc.copy_(src)
        torch.cuda.synchronize()
        log("[bench] traffic probe done: 3 prefill steps, 2 copies of 268435456 bytes")
        st.close()
        return

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

    # -------------------------------------------------------- warm prefill
    # Warm-up steps run with every launch timed: they give the per-kernel
    # breakdown and name the dominant kernel. The timed steps then bracket
    # only that kernel's launch site with events (events between
    # back-to-back kernels cost time of their own).
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

    hs.hs_stage_set_timing_sites(st.h, dom["site"])
    hs.hs_stage_set_timing(st.h, 1)
    ms_step = run_steps(args.steps)
    hs.hs_stage_set_timing(st.h, 0)
    hs.hs_stage_set_timing_sites(st.h, None)
    timed = [s for s in hs.hs_stage_read_timing(st.h)
             if s["name"] == dom["name"] and s["site"] == dom["site"]]
    assert timed and timed[0]["launches"] == args.steps * dom["launches"] // nw
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
    log(f"[bench] dominant kernel {dom['name']} ({dom['site']}): {dom_avg_s * 1e6:.1f} us, "
        f"{achieved:.0f} TFLOP/s in the timed steps")
    roofline = {"bound": "mfma", "kernel": dom["name"],
                "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic_from_profiles(dom["name"]),
                "flops_per_launch": dom_flops, "avg_launch_us": round(dom_avg_s * 1e6, 2)}
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)

    # ------------------------------------------------------------- decode
    i = prefill_once()
    xd = torch.empty((1, H), dtype=torch.bfloat16, device=dev)
    xd.copy_(x[:1])
    od = torch.empty((1, H), dtype=torch.bfloat16, device=dev)
    for _ in range(4):
        st.decode([i], xd.data_ptr(), od.data_ptr(), 0, sp)
    stream.synchronize()
    nd = args.decode_steps - 4
    ev0.record(stream)
    for _ in range(nd):
        st.decode([i], xd.data_ptr(), od.data_ptr(), 0, sp)
    ev1.record(stream)
    stream.synchronize()
    dec_ms = ev0.elapsed_time(ev1) / nd
    ctx = P + args.decode_steps
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
    imp = []
    for _ in range(reps):
        ev0.record(stream)
        hs.hs_kv_import(dst.h, blob.data_ptr(), size, sp)
        ev1.record(stream)
        stream.synchronize()
        imp.append(ev0.elapsed_time(ev1))
        hs.hs_seq_free(dst.h, i)
    imp_ms = statistics.median(imp)
    used = size - 256
    log(f"[bench] KV export {2 * used / (exp_ms / 1e3) / 1e9:.0f} GB/s, "
        f"import {2 * used / (imp_ms / 1e3) / 1e9:.0f} GB/s ({used / 1e6:.1f} MB)")
    dst.close()

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
        "cold_ttft_ms": round(t_cold * 1e3, 3),
        "cold_load_only_ms": round(t_load * 1e3, 3),
        "h2d_GBps": round(img.numel() / t_load / 1e9, 2),
        "h2d_frac_of_pcie": round(img.numel() / t_load / 1e9 / PEAK_PCIE_GBPS, 4),
        "overlap_efficiency": round((t_load + t_prefill - t_cold) / min(t_load, t_prefill), 3),
        "decode_ms_per_step": round(dec_ms, 4),
        "decode_tok_s": round(1e3 / dec_ms, 1),
        "decode_hbm_frac": round(dec_bytes / (dec_ms / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
        "kv_export_GBps": round(2 * used / (exp_ms / 1e3) / 1e9, 1),
        "kv_import_GBps": round(2 * used / (imp_ms / 1e3) / 1e9, 1),
    }
    st.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
