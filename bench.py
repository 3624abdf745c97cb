"""Benchmark: one step = one full pass of the tuning hot path on the ResNet-18
batch-1 conv set (12 layers, fp32 NCHW, 256 seeded candidates per layer,
128 from each of the two kernel families that apply: direct and fp32 MFMA):

  1. tune every layer at 25% of the CUs, as 4 concurrent clients on the 4
     disjoint 64-CU slots, which take the layers from one shared queue,
     largest first;
  2. the same at 50% (2 clients on 128-CU slots) and at 100% (1 client);
     each client screens every candidate (2 warm-up + 5 x 10 timed runs),
     re-measures its top 8 (21 x 10 runs, interleaved) and picks the winner;
  3. cross-evaluate each layer's three winners on all three shares (3 x 3).

value = candidates screened per second over the timed steps (whole job, one
GPU). The roofline object describes the best schedule of the 64->64 3x3
56x56 layer at 100% of the CUs: achieved TFLOP/s = its FLOPs / its latency,
where the latency is the median over 21 interleaved repeats of the mean of
10 back-to-back runs, timed with HIP events on its own stream inside the
timed region.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FRACTIONS = (0.25, 0.5, 1.0)
HEADLINE = "r18.2"


def runs_per_candidate(cfg, n_layers: int, n_fractions: int) -> float:
    """Convolution launches one step makes per screened candidate: the screen,
    the top-T re-measure and the cross-evaluation, over all layers and shares."""
    p1, p2 = cfg.stage1, cfg.stage2
    screen = cfg.n_candidates * (p1.warmup + p1.repeats * p1.launches)
    remeasure = cfg.top_t * (p2.warmup + p2.repeats * p2.launches)
    cross = n_fractions * n_fractions * (p2.warmup + p2.repeats * p2.launches)
    runs = n_layers * (n_fractions * (screen + remeasure) + cross)
    return runs / (n_layers * n_fractions * cfg.n_candidates)


def cpu_baseline(cfg, runs_per_cand: float, budget_s: float = 15.0) -> dict:
    """The fp64 oracle timed on this host on a bounded sample of the workload.

    One oracle convolution stands in for one convolution launch of the tuner, so
    candidates/s = oracle convolutions/s / (launches per screened candidate)."""
    import oracle
    from paper_2008_03602_amd import synth

    threads = len(os.sched_getaffinity(0))
    done, flops, t_total = 0, 0, 0.0
    # the layer list is walked round-robin until the time budget is used
    while t_total < budget_s:
        op = cfg.ops[done % len(cfg.ops)]
        x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), cfg.dist, cfg.seed, cfg.config_id,
                                 done % len(cfg.ops))
        t0 = time.perf_counter()
        oracle.conv2d(x, w, (op.stride_h, op.stride_w), (op.pad_h, op.pad_w), threads=threads)
        t_total += time.perf_counter() - t0
        flops += op.flops()
        done += 1
    convs = done / t_total
    return {"value": convs / runs_per_cand, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "oracle_convs_per_s": convs, "gflops": flops / t_total / 1e9, "seconds": t_total,
            "sample": "%d fp64 oracle convolutions at full size, the %d ResNet-18 b1 layers in turn "
                      "(%.1f passes over the list), %.1f s on %d threads; candidates/s = convolutions/s "
                      "divided by the %.1f convolution launches the GPU step makes per screened candidate"
                      % (done, len(cfg.ops), done / len(cfg.ops), t_total, threads, runs_per_cand)}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--candidates", type=int, default=None, help="override (default 256 per layer)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--report", default=None, help="write the full per-layer report (JSON) here")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the tuning clients share one device through CU masks; "
              "a second GPU is not used by this build (run with --gpus 1).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2008_03602_amd import _lib as L, tuner as T, workloads as W

    L.ct_init(0)
    cfg = W.config(2)
    if a.candidates:
        cfg.n_candidates = a.candidates
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops)]
    cands = T.sample_all(layers, cfg)
    n_per_step = sum(len(c) for c in cands.values()) * len(FRACTIONS)
    masks = [L.ct_cu_mask(f, 0) for f in FRACTIONS]

    def step():
        res = {f: T.tune_model_at_fraction(layers, cands, cfg, f) for f in FRACTIONS}
        cross = {}
        for ld in layers:
            winners = [next(r for r in res[f] if r.layer_id == ld.layer_id).winner for f in FRACTIONS]
            if all(wn is not None for wn in winners):
                cross[ld.op.name] = T.cross_eval(ld, winners, masks, cfg.stage2)
        return res, cross

    def progress(what, t):
        print("[bench] %s done in %.1f s" % (what, time.perf_counter() - t), file=sys.stderr, flush=True)

    for i in range(a.warmup):
        tw = time.perf_counter()
        step()
        progress("warm-up step %d/%d" % (i + 1, a.warmup), tw)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    steps = []
    for i in range(a.steps):
        ts = time.perf_counter()
        steps.append(step())
        progress("timed step %d/%d" % (i + 1, a.steps), ts)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    res, cross = steps[-1]

    value = n_per_step * a.steps / elapsed
    head = {f: next(r for r in res[f] if r.op.name == HEADLINE) for f in FRACTIONS}
    op = head[1.0].op
    per_fraction = []
    for f in FRACTIONS:
        r = head[f]
        tf = op.flops() / (r.winner_lat_us * 1e-6) / 1e12
        per_fraction.append({"fraction": f, "cus": int(round(256 * f)), "latency_us": r.winner_lat_us,
                             "tflops": tf, "frac_of_scaled_fp32_peak": tf / (T.PEAK_FP32_TFLOPS * f),
                             "schedule": T.describe_schedule(op, r.winner),
                             "kernel": L.ct_kernel_name(op, r.winner)})
    best_layer = []
    for f in FRACTIONS:
        for r in res[f]:
            if r.winner is None:
                continue
            tf = r.op.flops() / (r.winner_lat_us * 1e-6) / 1e12
            best_layer.append((tf / (T.PEAK_FP32_TFLOPS * f), tf, f, r.op.name))
    best_layer.sort(reverse=True)
    r100 = head[1.0]
    ach = op.flops() / (r100.winner_lat_us * 1e-6) / 1e12
    fr = {f: T.fraction_report(res[f]) for f in FRACTIONS}
    # HBM bytes per launch of this kernel and shape from committed counter
    # runs, if the kernel's sources are unchanged since they were taken
    from paper_2008_03602_amd import profsum
    tblk = profsum.find_traffic(os.path.join(ROOT, "profiles"), per_fraction[-1]["kernel"],
                                per_fraction[-1]["schedule"])
    line = {
        "metric": "tuning candidates measured/sec (1 GPU); best conv2d TFLOP/s and % roofline per CU fraction",
        "value": value, "unit": "candidates/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": elapsed / a.steps * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "ResNet-18 b1 conv set (12 layers) fp32 NCHW, %d seeded candidates per layer "
                               "(equal shares per kernel family), "
                               "tuned at 25/50/100%% CUs by 4/2/1 concurrent CU-masked clients sharing a "
                               "largest-first layer queue, then a 3x3 cross-evaluation of the winners" % cfg.n_candidates,
                   "candidates_per_step": n_per_step, "layers": len(layers), "seed": cfg.seed,
                   "protocol": {"screen": [cfg.stage1.warmup, cfg.stage1.repeats, cfg.stage1.launches],
                                "remeasure_top": cfg.top_t,
                                "remeasure": [cfg.stage2.warmup, cfg.stage2.repeats, cfg.stage2.launches]}},
        "per_fraction_throughput": {str(f): fr[f] for f in FRACTIONS},
        "roofline": {"bound": "mfma" if "igemm" in per_fraction[-1]["kernel"] else "alu",
                     "achieved": ach, "peak": T.PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / T.PEAK_FP32_TFLOPS,
                     "traffic": tblk["traffic_bytes"] if tblk else None,
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "algorithmic_bytes_per_launch": op.bytes_moved(),
                     "kernel": per_fraction[-1]["kernel"], "layer": HEADLINE,
                     "flops_per_launch": op.flops(), "latency_us": r100.winner_lat_us,
                     "launch_shape": per_fraction[-1]["schedule"]},
        "best_per_fraction": per_fraction,
        "best_layer_by_scaled_peak": {"layer": best_layer[0][3], "fraction": best_layer[0][2],
                                      "tflops": best_layer[0][1], "frac": best_layer[0][0]},
    }
    if a.report:
        rep = {"line": line, "fractions": {str(f): [r.summary() for r in res[f]] for f in FRACTIONS},
               "cross_eval": {k: v.tolist() for k, v in cross.items()}}
        with open(a.report, "w") as fh:
            json.dump(rep, fh, indent=1)
    if not a.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, runs_per_candidate(cfg, len(layers), len(FRACTIONS)))
    print(json.dumps(line), flush=True)
    torch.cuda.synchronize()
    L.ct_shutdown()  # release the library's streams and events before interpreter exit
    return 0


if __name__ == "__main__":
    sys.exit(main())
