#!/usr/bin/env python3
"""Throughput of CoFiE's evidence-selection path (NGFF + QER) on one MI355X.

One step is the whole path over one batch of the 1 fps workload: NGFF
(histograms, novelty scores, keep rule) over a 256-frame 448x448 RGB stream,
then QER (bf16 MFMA text-to-visual scores, per-frame aggregation, top-16)
over 128 candidate frames of 256 visual tokens with 32 query tokens, 28
heads, head dim 128.  Inputs are seeded synthetic data resident in HBM;
several copies are rotated so that the 256 MiB last-level cache cannot serve
a step from the previous one.

Prints one JSON line: whole-step frames/s, per-stage figures, the roofline
fraction of the dominant kernel (its duration measured live with HIP events
bracketing every kernel the library launches) and the CPU oracle's rate on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("NGFF frames/s (GB/s vs HBM peak); QER candidate frames ranked/s (MFMA util)")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_1fps_stream.md")
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--rotate", type=int, default=3, help="input copies cycled through")
    ap.add_argument("--mode", choices=["graph", "eager"], default="eager",
                    help="call the library eagerly, or replay the step as a captured HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="target wall time of the CPU oracle sample")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this build "
              "(the evidence-selection path runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_03675_amd import binding as B
    from paper_2609_03675_amd import synth

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)
    B.lib()
    cfg = 2
    wl = synth.WORKLOADS[cfg]
    n, H, W, C = wl.T, wl.H, wl.W, 3

    # ---- inputs (host generation, then resident copies in HBM) -------------------
    frames_np = synth.frames(cfg)
    Q_np, K_np, offs_np = synth.qer_inputs(cfg)
    frames = [torch.from_numpy(frames_np).cuda() for _ in range(args.rotate)]
    Kd = [torch.from_numpy(K_np.view(np.int16)).cuda().view(torch.bfloat16) for _ in range(args.rotate)]
    Qd = torch.from_numpy(Q_np.view(np.int16)).cuda().view(torch.bfloat16)
    offs = torch.from_numpy(offs_np).cuda()
    n_vis = K_np.shape[0]
    n_frames = offs_np.size - 1

    # retention threshold for the target kept count, calibrated once on the GPU
    rule0 = B.keep_rule(wl.hist_mode, 0.3, 30, 4)
    tau = B.cofie_ngff_calibrate(frames[0], wl.bins, rule0, wl.target)

    # preallocated outputs and scratch: the step allocates nothing
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    mask = torch.empty(n, dtype=torch.uint8, device="cuda")
    count = torch.empty(1, dtype=torch.int32, device="cuda")
    probe_rule = B.keep_rule(wl.hist_mode, 0.3, 30, 4)
    ngff_ws = torch.empty(B.ngff_workspace_bytes(n, H, W, C, wl.bins, probe_rule), dtype=torch.uint8,
                          device="cuda")
    rule = B.keep_rule(wl.hist_mode, 0.3, 30, 4, tau_per_segment=tau, out_count=count,
                       workspace=ngff_ws)
    desc = B.qer_desc(wl.n_q, n_vis, n_frames, wl.H_q, wl.H_kv, wl.d)
    qer_ws = torch.empty(B.qer_workspace_bytes(desc, wl.k_top), dtype=torch.uint8, device="cuda")
    w_out = torch.empty(n_frames, dtype=torch.float32, device="cuda")
    idx_out = torch.empty(wl.k_top, dtype=torch.int32, device="cuda")

    def step(i):
        r = i % args.rotate
        B.cofie_ngff_filter(frames[r], wl.bins, rule, out_scores=scores, out_mask=mask)
        B.cofie_qer_rank(Qd, Kd[r], offs, wl.k_top, out_scores=w_out, out_idx=idx_out,
                         workspace=qer_ws)

    for i in range(max(args.warmup, args.rotate)):
        step(i)
    torch.cuda.synchronize()
    kept = int(count.item())

    graphs = None
    if args.mode == "graph":
        graphs = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for r in range(args.rotate):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=side):
                    step(r)
                graphs.append(g)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        for i in range(args.warmup):
            graphs[i % args.rotate].replay()
        torch.cuda.synchronize()

    def run_steps(k):
        for i in range(k):
            if graphs is not None:
                graphs[i % args.rotate].replay()
            else:
                step(i)

    # ---- timed region ---------------------------------------------------------------
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t0.record()
    run_steps(args.steps)
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps

    # the other launch mode, for reference
    torch.cuda.synchronize()
    ms_step_other = None
    if graphs is not None:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(args.steps):
            step(i)
        e1.record()
        torch.cuda.synchronize()
        ms_step_other = e0.elapsed_time(e1) / args.steps

    # ---- per-kernel durations, live HIP events around every library launch ------------
    B.cofie_profiler_reset()
    B.cofie_profiler_enable(True)
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    B.cofie_profiler_enable(False)
    kern = {}
    for name in ("ngff_fill", "ngff_hist", "ngff_band_next", "ngff_select", "qer_fold",
                 "qer_score", "qer_frame_mean", "qer_topk"):
        ms, cnt = B.cofie_profiler_read(name)
        if cnt:
            kern[name] = {"avg_us": 1e3 * ms / cnt, "launches": cnt}
    B.cofie_profiler_reset()

    # attainable streaming bandwidth: a plain read and a plain copy of 1 GiB
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    sink = torch.empty(1 << 20, dtype=torch.int32, device="cuda")

    def timed(fn, reps=10):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(reps):
            fn()
        c1.record()
        torch.cuda.synchronize()
        return c0.elapsed_time(c1) * 1e-3 / reps

    read_gbs = (1 << 30) / timed(lambda: B.cofie_diag_stream_read(src, sink)) / 1e9
    copy_gbs = 2 * (1 << 30) / timed(lambda: B.cofie_diag_stream_copy(src, dst)) / 1e9
    del src, dst, sink

    # ---- algorithmic work per launch -------------------------------------------------------
    ngff_bytes = n * H * W * C                                   # every frame byte read once
    qer_bytes = n_vis * wl.H_kv * wl.d * 2 + wl.n_q * wl.H_q * wl.d * 2   # K once + Q
    qer_flops = 2.0 * wl.n_q * n_vis * wl.H_q * wl.d
    hist_us = kern["ngff_hist"]["avg_us"]
    score_us = kern["qer_score"]["avg_us"]
    ngff_gbs = ngff_bytes / (hist_us * 1e-6) / 1e9
    qer_gbs = qer_bytes / (score_us * 1e-6) / 1e9
    qer_tflops = qer_flops / (score_us * 1e-6) / 1e12
    ngff_stage_us = sum(v["avg_us"] for k, v in kern.items() if k.startswith("ngff"))
    qer_stage_us = sum(v["avg_us"] for k, v in kern.items() if k.startswith("qer"))
    if score_us >= hist_us:
        roof = {"kernel": "qer_score", "bound": "hbm", "achieved": round(qer_gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(qer_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("qer_score_kernel"), "algorithmic_bytes": qer_bytes,
                "avg_us": round(score_us, 2)}
    else:
        roof = {"kernel": "ngff_hist", "bound": "hbm", "achieved": round(ngff_gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ngff_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("ngff_hist_kernel"), "algorithmic_bytes": ngff_bytes,
                "avg_us": round(hist_us, 2)}

    # ---- CPU oracle on a bounded sample ------------------------------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, frames_np, Q_np, K_np, offs_np, float(tau[0].item()), args.cpu_seconds)

    value = n / (ms_step * 1e-3)
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8+bf16",
        "data": "synthetic",
        "config": {"workload": "1fps_stream", "frames": n, "H": H, "W": W, "hist_mode": wl.hist_mode,
                   "bins": wl.bins, "retain": wl.retain, "L_max": 30, "M_min": 4,
                   "qer": {"n_q": wl.n_q, "H_q": wl.H_q, "H_kv": wl.H_kv, "d": wl.d,
                           "candidates": n_frames, "tokens_per_frame": wl.tokens,
                           "k_top": wl.k_top, "dtype": "bf16", "score_mode": "logit"},
                   "step": args.mode, "rotated_copies": args.rotate},
        "roofline": roof,
        "cpu_baseline": cpu,
        "stages": {
            "ngff_frames_per_s": round(n / (ngff_stage_us * 1e-6), 1),
            "ngff_hist_GBps": round(ngff_gbs, 1),
            "ngff_hist_frac_hbm": round(ngff_gbs / HBM_PEAK_GBS, 4),
            "ngff_hist_traffic": measured_traffic("ngff_hist_kernel"),
            "qer_candidates_per_s": round(n_frames / (qer_stage_us * 1e-6), 1),
            "qer_score_GBps": round(qer_gbs, 1),
            "qer_score_frac_hbm": round(qer_gbs / HBM_PEAK_GBS, 4),
            "qer_score_TFLOPs": round(qer_tflops, 2),
            "qer_mfma_util": round(qer_tflops / BF16_PEAK_TFLOPS, 4),
            "kernels_us": {k: round(v["avg_us"], 2) for k, v in kern.items()},
            "kept_frames": kept,
            "ms_per_step_eager_when_graph": None if ms_step_other is None else round(ms_step_other, 5),
            "copy_probe_GBps": round(copy_gbs, 1),
            "read_probe_GBps": round(read_gbs, 1),
            "wall_s": round(wall, 3),
        },
    }
    print(json.dumps(out), flush=True)


def measured_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed PMC summary, or None
    when the summary is missing or the kernel's source changed since then."""
    import hashlib
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return None
    for line in lines:
        parts = line.split()
        if len(parts) == 5 and parts[0] == "traffic" and parts[1] == kernel:
            src = os.path.join(ROOT, "paper_2609_03675_amd", "csrc", parts[3])
            try:
                digest = hashlib.sha256(open(src).read().encode()).hexdigest()
            except OSError:
                return None
            return int(parts[2]) if digest == parts[4] else None
    return None


def cpu_baseline(wl, frames_np, Q_np, K_np, offs_np, tau, target_s):
    """The oracle, as it stands, on this host's cores: whole NGFF passes over
    the 256-frame stream and whole QER passes over the 128 candidates, each
    repeated for about half of the time budget; the step rate is the inverse
    of the two mean times added."""
    import oracle

    threads = oracle.num_threads()
    n = frames_np.shape[0]
    M = oracle.mass(oracle.PER_CHANNEL, wl.H, wl.W)

    def repeat(fn, budget):
        t0 = time.perf_counter()
        reps = 0
        while True:
            fn()
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget or reps >= 200:
                return el / reps, reps

    def ngff():
        h = oracle.histogram(frames_np, wl.bins, oracle.PER_CHANNEL)
        oracle.ngff_select(h, M, tau, 30, 4)

    def qer():
        w = oracle.qer_scores(Q_np, K_np, offs_np, wl.H_q, wl.H_kv, wl.d)
        oracle.topk(w, wl.k_top)

    ngff_s, r1 = repeat(ngff, 0.5 * target_s)
    qer_s, r2 = repeat(qer, 0.5 * target_s)
    step_s = ngff_s + qer_s
    return {"value": round(n / step_s, 3), "unit": "frames/s", "cores": threads, "kind": "oracle",
            "sample": f"full workload step: NGFF oracle on the {n}-frame stream x{r1} and the fp64 "
                      f"QER oracle on all {wl.n_frames} candidates x{r2}; rate = {n} frames / "
                      f"(mean NGFF time + mean QER time)",
            "ngff_s": round(ngff_s, 5), "qer_s": round(qer_s, 5)}


if __name__ == "__main__":
    main()
