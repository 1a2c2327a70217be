#!/usr/bin/env python3
"""Throughput of CoFiE's evidence-selection path (NGFF + QER) on one MI355X.

One step is the whole path over one batch of the multi-stream workload, the
largest one: NGFF (histograms, novelty scores, keep rule with a calibrated
threshold per stream) over 32 streams x 512 RGB frames of 448x448 (9.87 GB),
then QER for the 4 queries of every stream (128 queries of 32 text tokens,
28 heads, head dim 128, bf16): each query ranks its stream's NGFF candidates
up to its timestamp, 144 visual tokens per frame, top-16, all streams in one
cofie_qer_rank_streams call (every stream's keys read once).  Inputs are seeded
synthetic data resident in HBM (far larger than the 256 MiB last-level
cache, so no step is served from the previous one).

Prints one JSON line: whole-step frames/s, per-stage figures, the roofline
fraction of the dominant kernel (its duration measured live with the HIP event
pair that every kernel the library launches carries in its dispatch) and the CPU oracle's rate on a
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
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_multistream.md")
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--qer", choices=["one-launch", "per-stream"], default="one-launch",
                    help="QER of the step: every stream's queries in one cofie_qer_rank_streams call, or one "
                         "cofie_qer_rank_batched call per stream")
    ap.add_argument("--two-streams", action="store_true",
                    help="run each step's QER on a second HIP stream beside NGFF (a streaming pipeline: "
                         "QER of one batch while NGFF filters the next); the kernels then share HBM, so "
                         "the per-kernel rates and the roofline are those of the overlapped kernels")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target wall time of the CPU oracle sample (all host threads)")
    ap.add_argument("--configs", default="",
                    help="comma-separated workload ids (1-5): print a per-workload stage report "
                         "(one JSON line each) instead of the headline step")
    ap.add_argument("--report", default="", help="with --configs: also write a markdown table here")
    ap.add_argument("--ms-streams", type=int, default=32,
                    help="with --configs 5: streams whose queries are ranked (of 32)")
    ap.add_argument("--push-batch", type=int, default=64,
                    help="with --configs: frames per stream and push of the online NGFF pass")
    ap.add_argument("--signals", default="",
                    help="comma-separated workload ids (1-5): time NGFF with the Table 5 alternative signals "
                         "(low-res frame difference, dHash) on the workload's frames (one JSON line each)")
    ap.add_argument("--attn-qer", default="",
                    help="comma-separated workload ids (2-4): time the last-layer prefill attention "
                         "with QER from its QK^T tiles (one JSON line each) instead of the headline step")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the evidence-selection path runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_03675_amd import binding as B
    from paper_2609_03675_amd import synth

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    torch.cuda.set_device(0)
    B.lib()
    if args.configs:
        config_report(args, [int(c) for c in args.configs.split(",")])
        return
    if args.attn_qer:
        attn_qer_report(args, [int(c) for c in args.attn_qer.split(",")])
        return
    if args.signals:
        signals_report(args, [int(c) for c in args.signals.split(",")])
        return
    headline(args)


NGFF_KERNELS = ("ngff_fill", "ngff_hist", "ngff_keep", "ngff_band", "ngff_next", "ngff_select")
QER_KERNELS = ("qer_fold", "qer_qop", "qer_score", "qer_frame_mean", "qer_topk")


class MsQuery:
    """The QER inputs of one stream of the multi-stream workload, resident on
    the GPU: its candidates (the keep rule's frames up to the last query's
    timestamp), their keys, the stacked queries and each query's prefix."""

    def __init__(self, torch, B, synth, cfg, s, kept):
        wl = synth.WORKLOADS[cfg]
        stamps = synth.multistream_queries(cfg, s)
        cand = kept[kept <= stamps.max()]
        self.nf = np.array([int((kept <= ts).sum()) for ts in stamps], np.int32)
        K = synth.multistream_k(cfg, s, cand)
        Q = np.stack([synth.multistream_q(cfg, s, g) for g in range(len(stamps))])
        self.n_cand = int(cand.size)
        self.n_vis = int(K.shape[0])
        self.K = torch.from_numpy(K.view(np.int16)).cuda().view(torch.bfloat16)
        self.Q = torch.from_numpy(Q.view(np.int16)).cuda().view(torch.bfloat16)
        self.offs = torch.from_numpy(synth.frame_offsets(np.full(self.n_cand, wl.tokens))).cuda()
        self.k_top = wl.k_top
        desc = B.qer_desc(wl.n_q, self.n_vis, self.n_cand, wl.H_q, wl.H_kv, wl.d)
        self.ws = torch.empty(B.qer_batched_workspace_bytes(desc, len(stamps), wl.k_top), dtype=torch.uint8,
                              device="cuda")
        self.w = torch.empty((len(stamps), max(self.n_cand, 1)), dtype=torch.float32, device="cuda")
        self.idx = torch.empty((len(stamps), wl.k_top), dtype=torch.int32, device="cuda")

    def rank(self, B):
        B.cofie_qer_rank_batched(self.Q, self.K, self.offs, self.nf, self.k_top, out_scores=self.w,
                                 out_idx=self.idx, workspace=self.ws)


def upload_frames(torch, synth, cfg, keep_host=0):
    """Every frame of the workload in one device buffer, generated stream by
    stream on the host; the host frames of the first `keep_host` streams are
    returned for the CPU baseline."""
    wl = synth.WORKLOADS[cfg]
    frames = torch.empty((wl.n, wl.H, wl.W, 3), dtype=torch.uint8, device="cuda")
    kept_host = []
    for s in range(wl.n_streams):
        host = synth.StreamPlan(cfg, s).frames()
        frames[s * wl.T:(s + 1) * wl.T].copy_(torch.from_numpy(host))
        if s < keep_host:
            kept_host.append(host)
    return frames, kept_host


def headline(args):
    """The timed step on the multi-stream workload (module docstring)."""
    import torch

    from paper_2609_03675_amd import binding as B
    from paper_2609_03675_amd import synth

    cfg = 5
    wl = synth.WORKLOADS[cfg]
    S, T = wl.n_streams, wl.T
    n, H, W, C = wl.n, wl.H, wl.W, 3

    # ---- inputs: frames in HBM, per-stream thresholds calibrated once on the GPU ----------
    frames, host_frames = upload_frames(torch, synth, cfg, keep_host=0 if args.no_cpu_baseline else 4)
    rule0 = B.keep_rule(wl.hist_mode, 0.3, 30, 4, T)
    tau = B.cofie_ngff_calibrate(frames, wl.bins, rule0, wl.target)
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    mask = torch.empty(n, dtype=torch.uint8, device="cuda")
    count = torch.empty(S, dtype=torch.int32, device="cuda")
    ngff_ws = torch.empty(B.ngff_workspace_bytes(n, H, W, C, wl.bins, rule0), dtype=torch.uint8, device="cuda")
    rule = B.keep_rule(wl.hist_mode, 0.3, 30, 4, T, tau_per_segment=tau, out_count=count, workspace=ngff_ws)
    B.cofie_ngff_filter(frames, wl.bins, rule, out_scores=scores, out_mask=mask)
    torch.cuda.synchronize()
    # The keep rule's candidates are the same at every step (same frames, same
    # thresholds), so each query's prefix length, which the host passes to the
    # ranking call, is read once here from the GPU's mask; the keys of the
    # candidates stand in for the encoder's output and are resident in HBM.
    mask_np = mask.cpu().numpy()
    qs = [MsQuery(torch, B, synth, cfg, s, np.flatnonzero(mask_np[s * T:(s + 1) * T])) for s in range(S)]
    n_queries = sum(len(q.nf) for q in qs)
    ranked = int(sum(int(q.nf.sum()) for q in qs))          # candidate frames ranked per step
    k_bytes = sum(q.n_vis for q in qs) * wl.H_kv * wl.d * 2  # every stream's keys read once
    q_bytes = sum(q.Q.numel() for q in qs) * 2
    # flops of the contraction as issued: every query of a stream against all its keys
    qer_flops = sum(2.0 * len(q.nf) * wl.n_q * q.n_vis * wl.H_q * wl.d for q in qs)
    if args.qer == "one-launch":
        # every stream's keys, candidates and queries side by side: one call
        Kall = torch.cat([q.K for q in qs])
        Qall = torch.cat([q.Q for q in qs])
        base = np.concatenate([[0], np.cumsum([q.n_vis for q in qs])])
        offs_all = torch.from_numpy(np.concatenate(
            [[0]] + [synth.frame_offsets(np.full(q.n_cand, wl.tokens))[1:] + base[i] for i, q in enumerate(qs)]
        ).astype(np.int32)).cuda()
        lay = B.StreamsLayout([q.n_vis for q in qs], [q.n_cand for q in qs], [len(q.nf) for q in qs],
                              np.concatenate([q.nf for q in qs]))
        sdesc = B.qer_desc(wl.n_q, int(base[-1]), int(sum(q.n_cand for q in qs)), wl.H_q, wl.H_kv, wl.d)
        sws = torch.empty(B.qer_streams_workspace_bytes(sdesc, lay, wl.k_top), dtype=torch.uint8, device="cuda")
        w_all = torch.empty((n_queries, lay.max_frames), dtype=torch.float32, device="cuda")
        idx_all = torch.empty((n_queries, wl.k_top), dtype=torch.int32, device="cuda")
        for q in qs:  # the per-stream copies are not needed any more
            q.K = q.Q = None
        torch.cuda.empty_cache()

        def qer_step():
            B.cofie_qer_rank_streams(Qall, Kall, offs_all, lay, wl.k_top, out_scores=w_all, out_idx=idx_all,
                                     workspace=sws)
    else:
        def qer_step():
            for q in qs:
                q.rank(B)

    # default priority, like every stream here
    qer_stream = torch.cuda.Stream() if args.two_streams else torch.cuda.current_stream()

    def step(i):
        B.cofie_ngff_filter(frames, wl.bins, rule, out_scores=scores, out_mask=mask)
        with torch.cuda.stream(qer_stream):
            qer_step()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    kept = int(count.sum().item())

    # ---- timed region ---------------------------------------------------------------
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t0.record()
    qer_stream.wait_stream(torch.cuda.current_stream())
    for i in range(args.steps):
        step(i)
    torch.cuda.current_stream().wait_stream(qer_stream)
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps

    # ---- per-kernel durations, live HIP events carried by every library launch --------
    B.cofie_profiler_reset()
    B.cofie_profiler_enable(True)
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    B.cofie_profiler_enable(False)
    kern = {}
    for name in NGFF_KERNELS + QER_KERNELS:
        ms, cnt = B.cofie_profiler_read(name)
        if cnt:
            kern[name] = {"avg_us": 1e3 * ms / cnt, "per_step": cnt / args.steps,
                          "us_per_step": 1e3 * ms / args.steps}
    B.cofie_profiler_reset()

    # attainable streaming bandwidth: a plain read and a plain copy of 1 GiB
    read_gbs = read_probe_gbs(torch, B)
    copy_gbs = copy_probe_gbs(torch, B)

    # ---- algorithmic work ------------------------------------------------------------------
    ngff_bytes = n * H * W * C                  # every frame byte read once
    qer_bytes = k_bytes + q_bytes               # keys once + queries
    hist = kern["ngff_hist"]
    score = kern["qer_score"]
    ngff_gbs = ngff_bytes / (hist["us_per_step"] * 1e-6) / 1e9
    qer_gbs = qer_bytes / (score["us_per_step"] * 1e-6) / 1e9
    qer_tflops = qer_flops / (score["us_per_step"] * 1e-6) / 1e12
    ngff_stage_us = sum(v["us_per_step"] for k, v in kern.items() if k.startswith("ngff"))
    qer_stage_us = sum(v["us_per_step"] for k, v in kern.items() if k.startswith("qer"))
    # the dominant kernel: the largest share of the step's GPU time
    if score["us_per_step"] >= hist["us_per_step"]:
        per = score["per_step"]
        roof = {"kernel": "qer_score", "bound": "hbm", "achieved": round(qer_gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(qer_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("qer_score_kernel"), "algorithmic_bytes": round(qer_bytes / per),
                "launches_per_step": per, "avg_us": round(score["avg_us"], 2)}
    else:
        roof = {"kernel": "ngff_hist", "bound": "hbm", "achieved": round(ngff_gbs, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ngff_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic("ngff_hist_kernel"), "algorithmic_bytes": ngff_bytes,
                "launches_per_step": hist["per_step"], "avg_us": round(hist["avg_us"], 2)}

    # ---- CPU oracle on a bounded sample ------------------------------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline_multistream(wl, cfg, host_frames, args.cpu_seconds)

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
        "config": {"workload": "multistream", "streams": S, "frames_per_stream": T, "frames": n, "H": H, "W": W,
                   "hist_mode": wl.hist_mode, "bins": wl.bins, "retain": wl.retain, "L_max": 30, "M_min": 4,
                   "step": "QER on a second HIP stream beside NGFF" if args.two_streams else "NGFF, then QER",
                   "qer": {"queries": n_queries, "n_q": wl.n_q, "H_q": wl.H_q, "H_kv": wl.H_kv, "d": wl.d,
                           "tokens_per_frame": wl.tokens, "k_top": wl.k_top, "dtype": "bf16",
                           "score_mode": "logit", "candidates_ranked": ranked,
                           "calls": ("one cofie_qer_rank_streams over all streams" if args.qer == "one-launch"
                                     else "one cofie_qer_rank_batched per stream")}},
        "roofline": roof,
        "cpu_baseline": cpu,
        "stages": {
            "ngff_frames_per_s": round(n / (ngff_stage_us * 1e-6), 1),
            "ngff_us": round(ngff_stage_us, 1),
            "ngff_hist_GBps": round(ngff_gbs, 1),
            "ngff_hist_frac_hbm": round(ngff_gbs / HBM_PEAK_GBS, 4),
            "ngff_hist_traffic": measured_traffic("ngff_hist_kernel"),
            "qer_us": round(qer_stage_us, 1),
            "qer_candidates_ranked_per_s": round(ranked / (qer_stage_us * 1e-6), 1),
            "qer_key_bytes": k_bytes,
            "qer_score_GBps": round(qer_gbs, 1),
            "qer_score_frac_hbm": round(qer_gbs / HBM_PEAK_GBS, 4),
            "qer_score_TFLOPs": round(qer_tflops, 2),
            "qer_mfma_util": round(qer_tflops / BF16_PEAK_TFLOPS, 4),
            "kernels_us_per_step": {k: round(v["us_per_step"], 2) for k, v in kern.items()},
            "kernels_avg_us": {k: round(v["avg_us"], 2) for k, v in kern.items()},
            "kernel_launches_per_step": {k: v["per_step"] for k, v in kern.items()},
            "kept_frames": kept,
            "copy_probe_GBps": round(copy_gbs, 1),
            "read_probe_GBps": round(read_gbs, 1),
            "wall_s": round(wall, 3),
        },
    }
    print(json.dumps(out), flush=True)


def cpu_baseline_multistream(wl, cfg, host_frames, target_s):
    """The oracle, as it stands, on this host's cores: whole streams of the
    same workload (NGFF with the stream's calibrated threshold, then the fp64
    QER of the stream's 4 queries over its candidates), as many as fit the
    time budget, on all threads; then one stream on one thread.  Rates are
    frames per second of oracle time (threshold calibration and input
    generation untimed)."""
    import oracle
    from paper_2609_03675_amd import synth

    M = oracle.mass(oracle.PER_CHANNEL, wl.H, wl.W)

    def stream_s(s, frames):
        h = oracle.histogram(frames, wl.bins, oracle.PER_CHANNEL)
        t_ngff = time.perf_counter()
        _, tau = oracle.ngff_calibrate(h, M, wl.target, 30, 4)          # untimed
        t_cal = time.perf_counter() - t_ngff
        _, mask, _ = oracle.ngff_select(h, M, tau[0], 30, 4)
        kept = np.flatnonzero(mask)
        stamps = synth.multistream_queries(cfg, s)
        cand = kept[kept <= stamps.max()]
        t_gen = time.perf_counter()
        K = synth.multistream_k(cfg, s, cand)                            # untimed
        Qs = [synth.multistream_q(cfg, s, g) for g in range(len(stamps))]
        t_gen = time.perf_counter() - t_gen
        for g, ts in enumerate(stamps):
            nc = int((kept <= ts).sum())
            offs = synth.frame_offsets(np.full(nc, wl.tokens))
            oracle.topk(oracle.qer_scores(Qs[g], K[:nc * wl.tokens], offs, wl.H_q, wl.H_kv, wl.d), wl.k_top)
        return t_cal + t_gen

    def run(streams, frames_of):
        t = 0.0
        for s in streams:
            fr = frames_of(s)
            t0 = time.perf_counter()
            untimed = stream_s(s, fr)
            t += time.perf_counter() - t0 - untimed
        return t

    def frames_of(s):
        return host_frames[s] if s < len(host_frames) else synth.StreamPlan(cfg, s).frames()

    threads = oracle.num_threads()
    t_all, done = 0.0, 0
    while done < wl.n_streams and (done == 0 or t_all < target_s):
        t_all += run([done], frames_of)
        done += 1
    oracle.set_num_threads(1)
    try:
        t_one = run([0], frames_of)
    finally:
        oracle.set_num_threads(threads)
    return {"value": round(done * wl.T / t_all, 3), "unit": "frames/s", "cores": threads, "kind": "oracle",
            "sample": f"the first {done} of the 32 streams (each: NGFF over its {wl.T} frames, then the fp64 QER "
                      f"of its 4 queries over their candidate prefixes, top-{wl.k_top}); rate = frames / oracle "
                      f"time on {threads} threads (threshold calibration and input generation untimed)",
            "seconds": round(t_all, 3),
            "single_core": {"value": round(wl.T / t_one, 3), "unit": "frames/s", "cores": 1,
                            "sample": "stream 0 alone on one thread", "seconds": round(t_one, 3)}}



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


def read_probe_gbs(torch, B) -> float:
    """Plain streaming read of 1 GiB (the attainable HBM read rate)."""
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    sink = torch.empty(1 << 20, dtype=torch.int32, device="cuda")
    for _ in range(3):
        B.cofie_diag_stream_read(src, sink)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        B.cofie_diag_stream_read(src, sink)
    e1.record()
    torch.cuda.synchronize()
    return (1 << 30) / (e0.elapsed_time(e1) * 1e-3 / 10) / 1e9


def median_call_us(torch, fn, reps: int, warmup: int = 3) -> float:
    """GPU time per call of fn(i): `reps` calls enqueued back to back between two
    HIP events, three such runs, the median of their means (the host's launch
    latency stays outside, as in a pipeline that keeps the GPU fed)."""
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    runs = []
    for _ in range(3):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(reps):
            fn(i)
        b.record()
        torch.cuda.synchronize()
        runs.append(a.elapsed_time(b) * 1e3 / reps)
    return float(np.median(runs))


def profiled_kernels(torch, B, fn, reps: int) -> dict:
    """Average duration (us) of every library kernel over `reps` calls of fn(i)."""
    B.cofie_profiler_reset()
    B.cofie_profiler_enable(True)
    for i in range(reps):
        fn(i)
    torch.cuda.synchronize()
    B.cofie_profiler_enable(False)
    out = {}
    # names are matched as substrings: these are the kernels of the paths used
    for name in ("ngff_fill", "ngff_hist", "ngff_keep", "ngff_band", "ngff_next", "ngff_select", "qer_fold", "qer_score",
                 "qer_soft_stats", "qer_soft_merge", "qer_soft_score", "qer_frame_mean", "qer_topk", "attn_qer",
                 "attn_merge"):
        ms, cnt = B.cofie_profiler_read(name)
        if cnt:
            out[name] = round(1e3 * ms / cnt, 2)
    B.cofie_profiler_reset()
    return out


def config_report(args, cfgs):
    """Per-workload stage figures: NGFF frames/s and histogram GB/s against the
    HBM peak and the measured read ceiling, the retention reached, QER
    candidates/s, K GB/s and MFMA utilisation, and the CPU oracle's time on the
    same host bytes."""
    import torch
    import oracle
    from paper_2609_03675_amd import binding as B
    from paper_2609_03675_amd import synth

    probe = read_probe_gbs(torch, B)
    copy_probe = copy_probe_gbs(torch, B)
    modes = {"gray": oracle.GRAY, "per_channel": oracle.PER_CHANNEL, "joint3d": oracle.JOINT3D}
    rows = []
    for cfg in cfgs:
        wl = synth.WORKLOADS[cfg]
        n, H, W = wl.n, wl.H, wl.W
        frame_bytes = H * W * 3
        mode = modes[wl.hist_mode]
        M = oracle.mass(mode, H, W)
        seg = wl.T if wl.n_streams > 1 else 0
        # frames, generated stream by stream; the oracle's histograms are timed
        # on the same host bytes as they go by
        frames = torch.empty((n, H, W, 3), dtype=torch.uint8, device="cuda")
        cpu_hist_s = 0.0
        hists = []
        for st in range(wl.n_streams):
            plan = synth.StreamPlan(cfg, st)
            hs = []
            for c0 in range(0, wl.T, 128):
                c = min(128, wl.T - c0)
                host = plan.frames(c0, c)
                frames[st * wl.T + c0:st * wl.T + c0 + c].copy_(torch.from_numpy(host))
                t0 = time.perf_counter()
                hs.append(oracle.histogram(host, wl.bins, mode))
                cpu_hist_s += time.perf_counter() - t0
            hists.append(np.concatenate(hs))
            del host
        copies = [frames]
        if n * frame_bytes * 3 < (1 << 30):  # small inputs: rotate copies past the 256 MiB cache
            copies += [frames.clone() for _ in range(2)]
        rule0 = B.keep_rule(wl.hist_mode, 0.3, 30, 4, seg)
        tau = B.cofie_ngff_calibrate(frames, wl.bins, rule0, wl.target)
        tau_np = tau.cpu().numpy()
        t0 = time.perf_counter()
        for st in range(wl.n_streams):
            oracle.ngff_select(hists[st], M, float(tau_np[st]), 30, 4)
        cpu_sel_s = time.perf_counter() - t0
        del hists
        count = torch.empty(wl.n_streams, dtype=torch.int32, device="cuda")
        mask = torch.empty(n, dtype=torch.uint8, device="cuda")
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        ws = torch.empty(B.ngff_workspace_bytes(n, H, W, 3, wl.bins, rule0), dtype=torch.uint8,
                         device="cuda")
        rule = B.keep_rule(wl.hist_mode, 0.3, 30, 4, seg, tau_per_segment=tau, out_count=count,
                           workspace=ws)

        def ngff_call(i):
            B.cofie_ngff_filter(copies[i % len(copies)], wl.bins, rule, out_scores=scores, out_mask=mask)

        reps = 30 if n * frame_bytes < (1 << 30) else 10
        ngff_us = median_call_us(torch, ngff_call, reps)
        nk = profiled_kernels(torch, B, ngff_call, reps)
        online = online_ngff(torch, B, wl, frames, tau, args.push_batch, mask)
        kept = int(count.sum().item())
        hist_gbs = n * frame_bytes / (nk["ngff_hist"] * 1e-6) / 1e9
        row = {"workload": wl.name, "config": cfg,
               "ngff": {"frames": n, "us_per_call": round(ngff_us, 2),
                        "frames_per_s": round(n / (ngff_us * 1e-6), 1),
                        "call_GBps": round(n * frame_bytes / (ngff_us * 1e-6) / 1e9, 1),
                        "hist_GBps": round(hist_gbs, 1), "hist_frac_hbm": round(hist_gbs / HBM_PEAK_GBS, 4),
                        "hist_frac_read_probe": round(hist_gbs / probe, 4),
                        "kept": kept, "retention": round(kept / n, 4), "target_retention": wl.retain,
                        "kernels_us": nk, "oracle_s": round(cpu_hist_s + cpu_sel_s, 3),
                        "oracle_cores": oracle.num_threads(), "online": online}}
        mask_np = mask.cpu().numpy()
        seg_len = wl.T if wl.n_streams > 1 else 0
        cidx, cseg = B.cofie_mask_compact(mask, seg_len)
        compact_us = median_call_us(torch, lambda i: B.cofie_mask_compact(mask, seg_len, out_idx=cidx,
                                                                          out_seg_start=cseg), 30)
        del copies, frames, ws
        torch.cuda.empty_cache()

        if cfg != 5:
            row["qer"], gather = qer_single(torch, B, oracle, synth, wl, cfg, probe, copy_probe)
        else:
            row["qer"] = qer_multistream(torch, B, oracle, synth, wl, cfg, probe, mask_np, args.ms_streams)
            gather = None
        row["glue"] = {"compact_us": round(compact_us, 2), "gather": gather}
        row["read_probe_GBps"] = round(probe, 1)
        print(json.dumps(row), flush=True)
        rows.append(row)
    if args.report:
        write_report(args, rows, probe)


def online_ngff(torch, B, wl, frames, tau, batch, mask_one_shot):
    """The same streams pushed `batch` frames at a time through the online
    state and finished: GPU time of all pushes and the finish (state creation
    outside), median of three passes; the final mask must equal the one-shot
    filter's."""
    S, T = wl.n_streams, wl.T
    fr = frames.view(S, T, wl.H, wl.W, 3)
    rule = B.keep_rule(wl.hist_mode, 0.3, 30, 4, tau_per_segment=tau)
    scores = torch.empty((S, T), dtype=torch.float32, device="cuda")
    mask = torch.empty((S, T), dtype=torch.uint8, device="cuda")
    runs = []
    for _ in range(3):
        st = B.cofie_ngff_stream_create(S, wl.H, wl.W, 3, wl.bins, rule)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for t0 in range(0, T, batch):
            B.cofie_ngff_stream_push(st, fr, scores, mask, col=t0, b=min(batch, T - t0))
        B.cofie_ngff_stream_finish(st, mask, T)
        e1.record()
        torch.cuda.synchronize()
        B.cofie_ngff_stream_destroy(st)
        runs.append(e0.elapsed_time(e1) * 1e3)
    us = float(np.median(runs))
    same = bool(torch.equal(mask.view(-1), mask_one_shot))
    pushes = -(-T // batch)
    return {"batch": batch, "pushes": pushes, "us_total": round(us, 1), "us_per_push": round(us / pushes, 2),
            "frames_per_s": round(S * T / (us * 1e-6), 1), "equals_one_shot": same}


def qer_figures(calls, n_cand, total_us, kbytes, score_us, flops, flops_head, kernels, cpu_s, probe):
    gbs = kbytes / (score_us * 1e-6) / 1e9
    return {"calls": calls, "candidates": n_cand, "us_total": round(total_us, 2),
            "candidates_per_s": round(n_cand / (total_us * 1e-6), 1),
            "score_GBps": round(gbs, 1), "score_frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
            "score_frac_read_probe": round(gbs / probe, 4),
            "mfma_util_computed": round(flops / (score_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "per_head_TFLOPs": round(flops_head / (score_us * 1e-6) / 1e12, 1),
            "kernels_us_per_call": kernels, "oracle_s": round(cpu_s, 3)}


def copy_probe_gbs(torch, B) -> float:
    """Plain streaming copy of 1 GiB, bytes read + written per second."""
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    us = median_call_us(torch, lambda i: B.cofie_diag_stream_copy(src, dst), 10)
    return 2 * (1 << 30) / (us * 1e-6) / 1e9


def qer_single(torch, B, oracle, synth, wl, cfg, probe, copy_probe):
    """One ranking call over the workload's candidates; K rotated over enough
    copies to exceed 512 MiB (at most 8).  Then the glue after it: the keys of
    the selected frames gathered in chronological order (the shortened key
    sequence of Sec. 3.3), timed against the plain copy."""
    Q, K, offs = synth.qer_inputs(cfg)
    bf16 = wl.qk_dtype == "bf16"

    def dev(x):
        return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) if bf16 else torch.from_numpy(x).cuda()

    Qd = dev(Q)
    Kc = [dev(K)]
    ncopy = min(8, max(2, -(-(512 << 20) // K.nbytes)))
    Kc += [Kc[0].clone() for _ in range(ncopy - 1)]
    offs_d = torch.from_numpy(offs).cuda()
    desc = B.qer_desc(wl.n_q, K.shape[0], wl.n_frames, wl.H_q, wl.H_kv, wl.d, dtype=B.BF16 if bf16 else B.F32)
    qws = torch.empty(B.qer_workspace_bytes(desc, wl.k_top), dtype=torch.uint8, device="cuda")
    w_out = torch.empty(wl.n_frames, dtype=torch.float32, device="cuda")
    idx = torch.empty(wl.k_top, dtype=torch.int32, device="cuda")

    def call(i):
        B.cofie_qer_rank(Qd, Kc[i % len(Kc)], offs_d, wl.k_top, out_scores=w_out, out_idx=idx, workspace=qws)

    us = median_call_us(torch, call, 30)
    kern = profiled_kernels(torch, B, call, 30)
    t0 = time.perf_counter()
    oracle.topk(oracle.qer_scores(Q, K, offs, wl.H_q, wl.H_kv, wl.d), wl.k_top)
    cpu_s = time.perf_counter() - t0
    terms = 3 if (wl.H_q != wl.H_kv and bf16) else 1   # folded GQA carries q^ as three bf16 terms
    flops = 2.0 * wl.n_q * K.shape[0] * wl.H_kv * wl.d * terms
    flops_head = 2.0 * wl.n_q * K.shape[0] * wl.H_q * wl.d
    fig = qer_figures(1, wl.n_frames, us, K.nbytes + Q.nbytes, kern["qer_score"], flops, flops_head, kern,
                      cpu_s, probe)

    # SOFTMAX mode on the same inputs: two passes over K (statistics, then
    # probabilities), their merge, the frame means and the top-k
    sdesc = B.qer_desc(wl.n_q, K.shape[0], wl.n_frames, wl.H_q, wl.H_kv, wl.d, dtype=B.BF16 if bf16 else B.F32,
                       score_mode=B.SOFTMAX)
    sws = torch.empty(B.qer_workspace_bytes(sdesc, wl.k_top), dtype=torch.uint8, device="cuda")

    def scall(i):
        B.cofie_qer_rank(Qd, Kc[i % len(Kc)], offs_d, wl.k_top, out_scores=w_out, out_idx=idx, workspace=sws,
                         score_mode=B.SOFTMAX)

    sus = median_call_us(torch, scall, 20)
    skern = profiled_kernels(torch, B, scall, 20)
    passes_us = skern.get("qer_soft_stats", 0.0) + skern.get("qer_soft_score", 0.0)
    fig["softmax"] = {"us_per_call": round(sus, 2), "kernels_us": skern,
                      "passes_GBps": round(2 * K.nbytes / (passes_us * 1e-6) / 1e9, 1),
                      "passes_frac_hbm": round(2 * K.nbytes / (passes_us * 1e-6) / 8e12, 4),
                      "per_head_TFLOPs": round(2 * flops_head / (passes_us * 1e-6) / 1e12, 1)}

    cap = K.shape[0]
    dst = torch.empty_like(Kc[0])
    goffs = torch.empty(wl.k_top + 1, dtype=torch.int32, device="cuda")
    grows = torch.empty(cap, dtype=torch.int32, device="cuda")

    def gather(i):
        B.cofie_gather_frames(Kc[i % len(Kc)], offs_d, idx, dst=dst, out_offsets=goffs, out_rows=grows)

    gus = median_call_us(torch, gather, 30)
    rows = int(goffs[-1].item())
    moved = 2 * rows * (K.nbytes // K.shape[0])
    gbs = moved / (gus * 1e-6) / 1e9
    g = {"frames": int((idx >= 0).sum().item()), "rows": rows, "us": round(gus, 2), "GBps": round(gbs, 1),
         "frac_copy_probe": round(gbs / copy_probe, 4), "copy_probe_GBps": round(copy_probe, 1)}
    return fig, g


def qer_multistream(torch, B, oracle, synth, wl, cfg, probe, mask_np, n_streams):
    """Each query of the first n_streams streams ranks that stream's NGFF-kept
    frames up to the query time (its own call, K shared by the stream's queries)."""
    total_us = cpu_s = score_us = flops = 0.0
    n_cand = calls = kbytes = 0
    acc = {}
    bat_us = bat_score_us = 0.0
    bat_calls = 0
    bat_equal = True
    bat_soft_us = soft_single_us = soft_err = 0.0
    for st in range(min(n_streams, wl.n_streams)):
        kept = np.flatnonzero(mask_np[st * wl.T:(st + 1) * wl.T])
        stamps = synth.multistream_queries(cfg, st)
        last = kept[kept <= stamps.max()]
        K_all = synth.multistream_k(cfg, st, last)
        Kd = torch.from_numpy(K_all.view(np.int16)).cuda().view(torch.bfloat16)
        # the stream's queries in one call: K read once for all of them
        nfq = np.array([int((kept <= ts).sum()) for ts in stamps], np.int32)
        if len(last) and wl.n_q % 16 == 0:
            Qs = np.stack([synth.multistream_q(cfg, st, qi) for qi in range(len(stamps))])
            Qsd = torch.from_numpy(Qs.view(np.int16)).cuda().view(torch.bfloat16)
            offs_all = torch.from_numpy(synth.frame_offsets(np.full(len(last), wl.tokens))).cuda()
            kb = min(wl.k_top, len(last))

            def bcall(i, Qsd=Qsd, offs_all=offs_all, nfq=nfq, kb=kb):
                return B.cofie_qer_rank_batched(Qsd, Kd, offs_all, nfq, kb)

            def bcall_soft(i, Qsd=Qsd, offs_all=offs_all, nfq=nfq, kb=kb):
                return B.cofie_qer_rank_batched(Qsd, Kd, offs_all, nfq, kb, score_mode=B.SOFTMAX)

            bat_soft_us += median_call_us(torch, bcall_soft, 10)
            ws, _ = bcall_soft(0)
            # SOFTMAX: each query normalises over its own prefix, like a call
            # given only the prefix's keys (equal to rounding)
            for qi in range(len(stamps)):
                if nfq[qi]:
                    n = int(nfq[qi])

                    def call_soft(i, qi=qi, n=n, offs_all=offs_all, kb=kb):
                        return B.cofie_qer_rank(Qsd[qi], Kd[:n * wl.tokens], offs_all[:n + 1].contiguous(), kb,
                                                score_mode=B.SOFTMAX)

                    soft_single_us += median_call_us(torch, call_soft, 10)
                    w1, _ = call_soft(0)
                    rd = (w1 - ws[qi, :n]).abs().max() / w1.abs().max()
                    soft_err = max(soft_err, float(rd))
            bat_us += median_call_us(torch, bcall, 10)
            bat_score_us += profiled_kernels(torch, B, bcall, 10)["qer_score"]
            bat_calls += 1
            wb, _ = bcall(0)
            # bit-equal to single-query calls over the same keys (the score
            # kernel's work split depends on the key count)
            for qi in range(len(stamps)):
                if nfq[qi]:
                    w1, _ = B.cofie_qer_rank(Qsd[qi], Kd, offs_all[:nfq[qi] + 1].contiguous(), kb)
                    bat_equal &= bool(torch.equal(w1.view(torch.int32), wb[qi, :nfq[qi]].contiguous().view(torch.int32)))
            torch.cuda.synchronize()
        for qi, ts in enumerate(stamps):
            nc = int((kept <= ts).sum())
            if nc == 0:
                continue
            Q = synth.multistream_q(cfg, st, qi)
            Qd = torch.from_numpy(Q.view(np.int16)).cuda().view(torch.bfloat16)
            offs = synth.frame_offsets(np.full(nc, wl.tokens))
            offs_d = torch.from_numpy(offs).cuda()
            k = min(wl.k_top, nc)
            Ksl = Kd[:nc * wl.tokens]

            def call(i, Qd=Qd, Ksl=Ksl, offs_d=offs_d, k=k):
                B.cofie_qer_rank(Qd, Ksl, offs_d, k)

            total_us += median_call_us(torch, call, 10)
            kern = profiled_kernels(torch, B, call, 10)
            for name, v in kern.items():
                acc[name] = acc.get(name, 0.0) + v
            score_us += kern["qer_score"]
            t0 = time.perf_counter()
            oracle.topk(oracle.qer_scores(Q, K_all[:nc * wl.tokens], offs, wl.H_q, wl.H_kv, wl.d), k)
            cpu_s += time.perf_counter() - t0
            n_cand += nc
            calls += 1
            kbytes += nc * wl.tokens * wl.H_kv * wl.d * 2 + Q.nbytes
            flops += 2.0 * wl.n_q * nc * wl.tokens * wl.H_kv * wl.d
        del Kd
    kern = {name: round(v / max(calls, 1), 2) for name, v in acc.items()}
    out = qer_figures(calls, n_cand, total_us, kbytes, score_us, flops, flops, kern, cpu_s, probe)
    if bat_calls:
        out["batched"] = {"calls": bat_calls, "us_total": round(bat_us, 2),
                          "candidates_per_s": round(n_cand / (bat_us * 1e-6), 1),
                          "score_us_total": round(bat_score_us, 2),
                          "speedup_vs_one_call_per_query": round(total_us / bat_us, 3),
                          "scores_equal_one_call_per_query": bat_equal,
                          "softmax_us_total": round(bat_soft_us, 2),
                          "softmax_one_call_per_query_us_total": round(soft_single_us, 2),
                          "softmax_max_rel_diff_vs_prefix_calls": soft_err}
    return out


def attn_qer_report(args, cfgs):
    """The last layer's prefill attention with QER read from its QK^T tiles
    (cofie_attn_qer) on the candidate frames of workloads 2-4: whole-call time,
    per-kernel times, and the attention kernel's rate against the bf16 MFMA
    peak.  Algorithmic flops: 4 d H_q per (query, visible key) pair of the
    causal attention, L (L + 1) / 2 pairs per head; QER adds no pass of its
    own.  For reference, the separate ranking pass (cofie_qer_rank over the
    same text rows and visual keys) is timed too."""
    import torch

    from paper_2609_03675_amd import binding as B
    from paper_2609_03675_amd import synth

    for cfg in cfgs:
        wl = synth.WORKLOADS[cfg]
        L, vb, ve = synth.attn_layout(cfg)
        gen = torch.Generator(device="cuda")
        gen.manual_seed(2609_3675_000 + cfg)
        Q = torch.randn((L, wl.H_q, wl.d), generator=gen, device="cuda").to(torch.bfloat16)
        K = torch.randn((L, wl.H_kv, wl.d), generator=gen, device="cuda").to(torch.bfloat16)
        V = torch.randn((L, wl.H_kv, wl.d), generator=gen, device="cuda").to(torch.bfloat16)
        offs = torch.from_numpy(synth.frame_offsets(np.full(wl.n_frames, wl.tokens))).cuda()
        out = torch.empty_like(Q)
        w = torch.empty(wl.n_frames, dtype=torch.float32, device="cuda")
        idx = torch.empty(wl.k_top, dtype=torch.int32, device="cuda")
        ws = torch.empty(B.attn_qer_workspace_bytes(B.attn_desc(L, wl.H_q, wl.H_kv, wl.d, vb, ve, wl.n_frames)),
                         dtype=torch.uint8, device="cuda")

        def call(i):
            B.cofie_attn_qer(Q, K, V, offs, vb, ve, wl.k_top, out=out, out_scores=w, out_idx=idx, workspace=ws)

        us = median_call_us(torch, call, 5, warmup=2)
        kern = profiled_kernels(torch, B, call, 5)
        Qt = torch.cat([Q[:vb], Q[ve:]]).contiguous()
        Kv = K[vb:ve].contiguous()

        def sep(i):
            B.cofie_qer_rank(Qt, Kv, offs, wl.k_top)

        sep_us = median_call_us(torch, sep, 10)
        flops = 4.0 * wl.d * wl.H_q * L * (L + 1) / 2
        tf = flops / (kern["attn_qer"] * 1e-6) / 1e12
        print(json.dumps({
            "workload": wl.name, "L": L, "visual_tokens": ve - vb, "text_tokens": L - (ve - vb),
            "H_q": wl.H_q, "H_kv": wl.H_kv, "d": wl.d, "frames": wl.n_frames, "k_top": wl.k_top,
            "us_per_call": round(us, 1), "kernels_us": kern,
            "roofline": {"kernel": "attn_qer", "bound": "mfma", "achieved": round(tf, 1),
                         "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(tf / BF16_PEAK_TFLOPS, 4),
                         "algorithmic_flops": flops},
            "separate_qer_rank_us": round(sep_us, 1)}), flush=True)
        del Q, K, V, out, ws, Qt, Kv
        torch.cuda.empty_cache()


def signals_report(args, cfgs):
    """NGFF with the alternative pre-encoder signals of the filtering-signal
    ablation (Table 5: low-res frame difference on a 32 x 32 grid, dHash) in
    place of the histogram, on a workload's frames: thresholds calibrated for
    the workload's retention, then the whole filter timed; the signature
    kernel's rate against the HBM peak (algorithmic bytes: every frame byte
    read once)."""
    import torch

    from paper_2609_03675_amd import binding as B
    from paper_2609_03675_amd import synth

    probe = read_probe_gbs(torch, B)
    for cfg in cfgs:
        wl = synth.WORKLOADS[cfg]
        frames, _ = upload_frames(torch, synth, cfg)
        n = wl.n
        seg = wl.T if wl.n_streams > 1 else 0
        fbytes = n * wl.H * wl.W * 3
        out = {"workload": wl.name, "frames": n, "read_probe_GBps": round(probe, 1)}
        for name, mode, G in (("framediff", B.FRAMEDIFF, 32), ("dhash", B.DHASH, 8)):
            rule0 = B.keep_rule(mode, 0.3, 30, 4, seg)
            tau = B.cofie_ngff_calibrate(frames, G, rule0, wl.target)
            count = torch.empty(wl.n_streams, dtype=torch.int32, device="cuda")
            ws = torch.empty(B.ngff_workspace_bytes(n, wl.H, wl.W, 3, G, rule0), dtype=torch.uint8, device="cuda")
            rule = B.keep_rule(mode, 0.3, 30, 4, seg, tau_per_segment=tau, out_count=count, workspace=ws)
            scores = torch.empty(n, dtype=torch.float32, device="cuda")
            mask = torch.empty(n, dtype=torch.uint8, device="cuda")

            def call(i, rule=rule, G=G, scores=scores, mask=mask):
                B.cofie_ngff_filter(frames, G, rule, out_scores=scores, out_mask=mask)

            reps = 10 if fbytes > (1 << 30) else 30
            us = median_call_us(torch, call, reps)
            B.cofie_profiler_reset()
            B.cofie_profiler_enable(True)
            for i in range(reps):
                call(i)
            torch.cuda.synchronize()
            B.cofie_profiler_enable(False)
            ms, cnt = B.cofie_profiler_read("ngff_sig")
            B.cofie_profiler_reset()
            sig_us = 1e3 * ms / max(cnt, 1)
            gbs = fbytes / (sig_us * 1e-6) / 1e9
            out[name] = {"grid": G if name == "framediff" else "8x9", "us_per_call": round(us, 1),
                         "frames_per_s": round(n / (us * 1e-6), 1), "signature_us": round(sig_us, 1),
                         "signature_GBps": round(gbs, 1), "signature_frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
                         "kept": int(count.sum().item()), "target_retention": wl.retain}
            del ws
        print(json.dumps(out), flush=True)
        del frames
        torch.cuda.empty_cache()


def write_report(args, rows, probe):
    cmd = f"python bench.py --configs {args.configs} --report {args.report}"
    lines = ["# Per-workload stage throughput (NGFF and QER) on one MI355X", "",
             "Command (from the repository root):", "", "```", cmd, "```", "",
             f"Read-probe ceiling (plain 1 GiB streaming read): {probe:.0f} GB/s.  HBM peak 8000 GB/s.  "
             "Call times: calls enqueued back to back between two HIP events (median of three runs); kernel times are averages of the "
             "library's per-kernel HIP-event profiler.  NGFF inputs under 1 GiB are rotated over three "
             "copies and K over enough copies to exceed 512 MiB, so the 256 MiB last-level cache cannot "
             "serve a call from the previous one.  The oracle columns time the CPU oracle on the same host "
             "bytes (all host cores).", "", "## NGFF", "",
             "| workload | frames | µs / call | frames/s | hist GB/s | % of 8 TB/s | % of read probe | "
             "kept (retention; target) | oracle s (threads) |",
             "|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        g = r["ngff"]
        lines.append(f"| {r['workload']} | {g['frames']} | {g['us_per_call']:.1f} | {g['frames_per_s']:,.0f} | "
                     f"{g['hist_GBps']:.0f} | {100 * g['hist_frac_hbm']:.1f} | "
                     f"{100 * g['hist_frac_read_probe']:.1f} | {g['kept']} ({g['retention']:.3f}; "
                     f"{g['target_retention']}) | {g['oracle_s']:.2f} ({g['oracle_cores']}) |")
    lines += ["", "Online NGFF (`cofie_ngff_stream_push` of every stream, then `cofie_ngff_stream_finish`; "
              "GPU time of the whole stream, state creation outside):", "",
              "| workload | frames per push and stream | pushes | µs per push | frames/s | final mask equals one-shot |",
              "|---|---|---|---|---|---|"]
    for r in rows:
        o = r["ngff"]["online"]
        lines.append(f"| {r['workload']} | {o['batch']} | {o['pushes']} | {o['us_per_push']:.1f} | "
                     f"{o['frames_per_s']:,.0f} | {o['equals_one_shot']} |")
    lines += ["", "## QER", "",
              "| workload | calls | candidates | µs total | candidates/s | score GB/s | % of 8 TB/s | "
              "% of read probe | MFMA util | per-head TFLOP/s | oracle s |",
              "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        q = r["qer"]
        lines.append(f"| {r['workload']} | {q['calls']} | {q['candidates']} | {q['us_total']:.1f} | "
                     f"{q['candidates_per_s']:,.0f} | {q['score_GBps']:.0f} | {100 * q['score_frac_hbm']:.1f} | "
                     f"{100 * q['score_frac_read_probe']:.1f} | {100 * q['mfma_util_computed']:.2f} % | "
                     f"{q['per_head_TFLOPs']:.1f} | {q['oracle_s']:.2f} |")
    soft = [r for r in rows if r["qer"].get("softmax")]
    if soft:
        lines += ["", "SOFTMAX mode (same inputs; per-head row softmax over the visual keys, head mean, then "
                  "Eq. 7): two passes over K.  GB/s counts 2·K over the two pass kernels' time; per-head TFLOP/s "
                  "counts 2·2·n_q·n_vis·H_q·d over the same time.", "",
                  "| workload | µs per call | pass 1 µs | merge µs | pass 2 µs | frame mean + top-k µs | "
                  "passes GB/s | % of 8 TB/s | per-head TFLOP/s |", "|---|---|---|---|---|---|---|---|---|"]
        for r in soft:
            sm = r["qer"]["softmax"]
            k = sm["kernels_us"]
            lines.append(f"| {r['workload']} | {sm['us_per_call']:.1f} | {k.get('qer_soft_stats', 0):.1f} | "
                         f"{k.get('qer_soft_merge', 0):.1f} | {k.get('qer_soft_score', 0):.1f} | "
                         f"{k.get('qer_frame_mean', 0) + k.get('qer_topk', 0):.1f} | {sm['passes_GBps']:.0f} | "
                         f"{100 * sm['passes_frac_hbm']:.1f} | {sm['per_head_TFLOPs']:.1f} |")
    for r in rows:
        b = r["qer"].get("batched")
        if b:
            lines += ["", f"{r['workload']}, the queries of each stream in one `cofie_qer_rank_batched` call (K read "
                      f"once per stream): {b['calls']} calls, {b['us_total']:.1f} µs total "
                      f"({b['candidates_per_s']:,.0f} candidates/s, {b['speedup_vs_one_call_per_query']:.2f}x one call "
                      f"per query; score kernels {b['score_us_total']:.1f} µs); scores equal to one call per query, "
                      f"bit for bit: {b['scores_equal_one_call_per_query']}.  SOFTMAX mode (each query's softmax "
                      f"over its own prefix): {b['softmax_us_total']:.1f} µs total in the same {b['calls']} calls, against "
                      f"{b['softmax_one_call_per_query_us_total']:.1f} µs for one call per query given its prefix's keys "
                      f"({b['softmax_one_call_per_query_us_total'] / b['softmax_us_total']:.2f}x); largest relative "
                      f"difference between the two {b['softmax_max_rel_diff_vs_prefix_calls']:.1e}."]
    lines += ["", "## Glue", "",
              "| workload | compaction µs | gathered frames | rows | gather µs | gather GB/s (read + write) | "
              "% of copy probe |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        g = r["glue"]
        ga = g["gather"]
        if ga:
            lines.append(f"| {r['workload']} | {g['compact_us']:.1f} | {ga['frames']} | {ga['rows']} | {ga['us']:.1f} | "
                         f"{ga['GBps']:.0f} | {100 * ga['frac_copy_probe']:.1f} |")
        else:
            lines.append(f"| {r['workload']} | {g['compact_us']:.1f} | | | | | |")
    lines += ["", "Compaction: `cofie_mask_compact` of the NGFF mask.  Gather: `cofie_gather_frames` of the keys "
              "of the QER-selected frames (chronological), bytes read + written.", ""]
    lines += ["", "MFMA utilisation = MFMA flops issued (the folded contraction; three bf16 query terms for "
              "grouped-query attention) / score-kernel time / 2.5 PFLOP/s.  Per-head TFLOP/s counts the "
              "per-head form 2·n_q·n_vis·H_q·d.", "", "Kernel times (µs per call):", ""]
    for r in rows:
        lines.append(f"- {r['workload']}: NGFF {r['ngff']['kernels_us']}; QER {r['qer']['kernels_us_per_call']}")
    with open(args.report, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
