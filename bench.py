"""Benchmark of the tuning hot path on the ResNet-18 batch-1 conv set.

Workload: the 12 distinct ResNet-18 b1 conv layers (fp32 NCHW, U(-1,1) inputs,
seed 0) with their 256-candidate seeded samples (128 per kernel family that
applies: direct and fp32 MFMA), tuned at 25 %, 50 % and 100 % of the CUs.

One step = one pass of the whole path over one batch of candidates: the
sample of every layer is cut into 8 fixed batches of 32 consecutive sample
positions (each batch holds 16 per family, as the sample interleaves them),
and step s takes batch s mod 8 of every layer:

  1. at 25 % of the CUs, 4 concurrent clients on the 4 disjoint 64-CU slots
     take the 12 layers from one shared queue, largest first; each screens the
     layer's 32 candidates (2 warm-up + 5 x 10 timed runs, HIP events on its
     CU-masked stream), re-measures its top 8 (21 x 10 runs, interleaved) and
     picks the winner with the tie rule;
  2. the same at 50 % (2 clients on 128-CU slots) and at 100 % (1 client);
  3. each layer's three winners are cross-evaluated on all three shares (3x3).

Eight consecutive steps cover the whole 256-candidate sample of every layer.

value = candidates screened per second over the timed steps (whole job, one
GPU). per_fraction_throughput: candidates/s of each share's runs over the
timed steps, from the library's per-client figures, and the 4 x 25 % against
1 x 100 % ratio. roofline: the fastest schedule that won the 64->64 3x3 56x56
layer at 100 % in a timed step; achieved TFLOP/s = its FLOPs / the median of
its stage-2 latencies (median over 21 interleaved repeats of the mean of 10
back-to-back runs, HIP events on its own stream) in the timed steps it won.

A wall-clock guard stops starting steps once the run has used --budget-s
seconds; the line then reports the steps actually timed.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

T_START = time.perf_counter()
ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FRACTIONS = (0.25, 0.5, 1.0)
HEADLINE = "r18.2"
SLICE = 32


def launches_per_candidate(cfg, n_layers: int, n_fractions: int, slice_n: int) -> float:
    """Convolution launches one step makes per screened candidate: the screen,
    the top-T re-measure and the cross-evaluation, over all layers and shares."""
    p1, p2 = cfg.stage1, cfg.stage2
    screen = slice_n * (p1.warmup + p1.repeats * p1.launches)
    remeasure = min(cfg.top_t, slice_n) * (p2.warmup + p2.repeats * p2.launches)
    cross = n_fractions * n_fractions * (p2.warmup + p2.repeats * p2.launches)
    runs = n_layers * (n_fractions * (screen + remeasure) + cross)
    return runs / (n_layers * n_fractions * slice_n)


def cpu_baseline(cfg, runs_per_cand: float, budget_s: float = 10.0, single_budget_s: float = 8.0) -> dict:
    """The fp64 oracle timed on this host on a bounded sample of the workload,
    on every core of the process's affinity set and on one thread.

    One oracle convolution stands in for one convolution launch of the tuner, so
    candidates/s = oracle convolutions/s / (launches per screened candidate)."""
    import oracle
    from paper_2008_03602_amd import synth

    def timed(threads: int, budget: float):
        done, flops, t_total = 0, 0, 0.0
        # the layer list is walked round-robin until the time budget is used
        while t_total < budget:
            op = cfg.ops[done % len(cfg.ops)]
            x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), cfg.dist, cfg.seed, cfg.config_id,
                                     done % len(cfg.ops))
            t0 = time.perf_counter()
            oracle.conv2d(x, w, (op.stride_h, op.stride_w), (op.pad_h, op.pad_w), threads=threads)
            t_total += time.perf_counter() - t0
            flops += op.flops()
            done += 1
        return done, flops, t_total

    threads = len(os.sched_getaffinity(0))
    done, flops, t_total = timed(threads, budget_s)
    d1, f1, t1 = timed(1, single_budget_s)
    convs = done / t_total
    return {"value": convs / runs_per_cand, "unit": "candidates/s", "cores": threads, "kind": "oracle",
            "oracle_convs_per_s": convs, "gflops": flops / t_total / 1e9, "seconds": t_total,
            "single_thread": {"value": d1 / t1 / runs_per_cand, "cores": 1, "oracle_convs_per_s": d1 / t1,
                              "gflops": f1 / t1 / 1e9, "seconds": t1, "convolutions": d1},
            "sample": "%d fp64 oracle convolutions at full size on %d threads (%.1f s) and %d on one thread "
                      "(%.1f s), the %d ResNet-18 b1 layers in turn; candidates/s = convolutions/s divided by "
                      "the %.1f convolution launches the GPU step makes per screened candidate"
                      % (done, threads, t_total, d1, t1, len(cfg.ops), runs_per_cand)}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--budget-s", type=float, default=420.0,
                    help="stop starting steps once the run has used this many seconds")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--uniform", action="store_true",
                    help="sample each layer's 256 candidates uniformly from its whole valid space "
                         "(no equal shares per kernel family)")
    ap.add_argument("--report", default=None, help="write the per-step, per-layer report (JSON) here")
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
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops)]
    full = T.sample_all(layers, cfg, uniform=a.uniform)
    n_batches = max(1, (cfg.n_candidates + SLICE - 1) // SLICE)
    masks = [L.ct_cu_mask(f, 0) for f in FRACTIONS]

    def step_cands(s: int):
        b = s % n_batches
        return {k: v[b * SLICE:(b + 1) * SLICE] for k, v in full.items()}

    def step(s: int):
        cands = step_cands(s)
        res = {f: T.tune_model_at_fraction(layers, cands, cfg, f) for f in FRACTIONS}
        cross = {}
        for ld in layers:
            winners = [next(r for r in res[f] if r.layer_id == ld.layer_id).winner for f in FRACTIONS]
            if all(wn is not None for wn in winners):
                cross[ld.op.name] = T.cross_eval(ld, winners, masks, cfg.stage2)
        return {"batch": s % n_batches, "res": res, "cross": cross,
                "screened": sum(len(c) for c in cands.values()) * len(FRACTIONS)}

    def log(msg):
        print("[bench] %s (%.1f s since start)" % (msg, time.perf_counter() - T_START), file=sys.stderr, flush=True)

    log("set-up done: %d layers, %d candidates each, %d batches of %d" % (len(layers), cfg.n_candidates,
                                                                          n_batches, SLICE))
    s = 0
    for i in range(a.warmup):
        tw = time.perf_counter()
        step(s)
        s += 1
        log("warm-up step %d/%d done in %.1f s" % (i + 1, a.warmup, time.perf_counter() - tw))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    steps = []
    for i in range(a.steps):
        if time.perf_counter() - T_START > a.budget_s:
            log("budget of %.0f s used: stopping after %d timed steps" % (a.budget_s, len(steps)))
            break
        ts = time.perf_counter()
        steps.append(step(s))
        s += 1
        log("timed step %d/%d (batch %d) done in %.1f s" % (i + 1, a.steps, steps[-1]["batch"],
                                                              time.perf_counter() - ts))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    if not steps:
        print("bench.py: no step was timed (budget used by the warm-up)", file=sys.stderr)
        return 1
    n_steps = len(steps)
    value = sum(st["screened"] for st in steps) / elapsed

    # per share: candidates and makespans of every timed step's run at that share
    per_fraction = {}
    for f in FRACTIONS:
        n = sum(sum(len(r.candidates) for r in st["res"][f]) for st in steps)
        sec = sum(T.fraction_report(st["res"][f])["seconds"] for st in steps)
        clients = T.fraction_report(steps[-1]["res"][f])["clients"]
        per_fraction[str(f)] = {"candidates": n, "seconds": sec, "candidates_per_s": n / sec, "clients": clients,
                                "cus_per_client": int(round(256 * f))}
    ratio = per_fraction["0.25"]["candidates_per_s"] / per_fraction["1.0"]["candidates_per_s"]

    # the roofline kernel: the fastest 100 % winner of the headline layer
    op = next(ld.op for ld in layers if ld.op.name == HEADLINE)
    wins = {}
    for st in steps:
        r = next(r for r in st["res"][1.0] if r.op.name == HEADLINE)
        if r.winner is not None:
            key = L.schedule_tuple(r.winner)
            wins.setdefault(key, {"sched": r.winner, "lat": []})["lat"].append(r.winner_lat_us)
    best_key = min(wins, key=lambda k: statistics.median(wins[k]["lat"]))
    best = wins[best_key]
    lat_us = statistics.median(best["lat"])
    ach = op.flops() / (lat_us * 1e-6) / 1e12
    desc = T.describe_schedule(op, best["sched"])
    kname = L.ct_kernel_name(op, best["sched"])
    # HBM bytes per launch of this kernel and shape from committed counter
    # runs, if the kernel's sources are unchanged since they were taken
    from paper_2008_03602_amd import profsum
    tblk = profsum.find_traffic(os.path.join(ROOT, "profiles"), kname, desc)

    # best schedule per share of the headline layer, and the best layer by scaled peak
    best_per_fraction = []
    for f in FRACTIONS:
        lats = {}
        for st in steps:
            r = next(r for r in st["res"][f] if r.op.name == HEADLINE)
            if r.winner is not None:
                lats.setdefault(L.schedule_tuple(r.winner), (r.winner, []))[1].append(r.winner_lat_us)
        k = min(lats, key=lambda k: statistics.median(lats[k][1]))
        lt = statistics.median(lats[k][1])
        tf = op.flops() / (lt * 1e-6) / 1e12
        best_per_fraction.append({"fraction": f, "cus": int(round(256 * f)), "latency_us": lt, "tflops": tf,
                                  "frac_of_scaled_fp32_peak": tf / (T.PEAK_FP32_TFLOPS * f),
                                  "kernel": L.ct_kernel_name(op, lats[k][0]),
                                  "knobs": list(T.describe_schedule(op, lats[k][0])["knobs"].values())})
    best_layer = max(((r.op.flops() / (r.winner_lat_us * 1e-6) / 1e12 / (T.PEAK_FP32_TFLOPS * f), f, r.op.name)
                      for st in steps for f in FRACTIONS for r in st["res"][f] if r.winner is not None))
    # where the screening time goes: per kernel family, the summed screened
    # latency x launches per candidate (stage 1, every share, timed steps)
    p1 = cfg.stage1
    runs1 = p1.warmup + p1.repeats * p1.launches
    fam_s = {}
    for st in steps:
        for f in FRACTIONS:
            for r in st["res"][f]:
                for c, lt, sc in zip(r.candidates, r.lat1, r.status1):
                    if sc == 0 and np.isfinite(lt):
                        k = W.FAMILY_NAMES[int(c.family)]
                        fam_s[k] = fam_s.get(k, 0.0) + float(lt) * 1e-6 * runs1
    tot_s = sum(fam_s.values()) or 1.0
    diag_ok = 0
    diag_n = 0
    for st in steps:
        for M in st["cross"].values():
            M = np.asarray(M)
            for g in range(M.shape[1]):
                diag_n += 1
                diag_ok += int(M[g, g] <= 1.03 * M[:, g].min())

    line = {
        "metric": "tuning candidates measured/sec (1 GPU); best conv2d TFLOP/s and % roofline per CU fraction",
        "value": value, "unit": "candidates/s", "n_gpus": 1, "steps": n_steps, "warmup": a.warmup,
        "ms_per_step": elapsed / n_steps * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "ResNet-18 b1 conv set (12 layers) fp32 NCHW, 256 seeded candidates per layer "
                               "(%s) in 8 fixed batches of 32; one step = one batch of "
                               "every layer tuned at 25/50/100%% CUs by 4/2/1 concurrent CU-masked clients sharing "
                               "a largest-first layer queue (screen, top-%d re-measure, tie rule), then a 3x3 "
                               "cross-evaluation of the winners"
                               % ("uniform over the valid space" if a.uniform else "equal shares per kernel family",
                                  cfg.top_t),
                   "candidates_per_step": steps[0]["screened"], "layers": len(layers), "seed": cfg.seed,
                   "batches_timed": sorted({st["batch"] for st in steps}),
                   "steps_requested": a.steps,
                   "protocol": {"screen": [cfg.stage1.warmup, cfg.stage1.repeats, cfg.stage1.launches],
                                "remeasure_top": cfg.top_t,
                                "remeasure": [cfg.stage2.warmup, cfg.stage2.repeats, cfg.stage2.launches]}},
        "per_fraction_throughput": per_fraction,
        "four_clients_25pct_vs_one_client_100pct": ratio,
        "roofline": {"bound": "mfma" if "igemm" in kname else "alu",
                     "achieved": ach, "peak": T.PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / T.PEAK_FP32_TFLOPS,
                     "traffic": tblk["traffic_bytes"] if tblk else None,
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "algorithmic_bytes_per_launch": op.bytes_moved(),
                     "kernel": kname, "layer": HEADLINE, "flops_per_launch": op.flops(), "latency_us": lat_us,
                     "timed_steps_won": len(best["lat"]), "launch_shape": desc},
        "best_per_fraction": best_per_fraction,
        "scaled_peak_target_met": {str(b["fraction"]): b["frac_of_scaled_fp32_peak"] >= 0.5
                                   for b in best_per_fraction},
        "best_layer_by_scaled_peak": {"layer": best_layer[2], "fraction": best_layer[1], "frac": best_layer[0]},
        "cross_eval_diagonal_within_3pct": [diag_ok, diag_n],
        "stage1_device_seconds_by_family": {k: {"seconds": v, "share": v / tot_s} for k, v in sorted(fam_s.items())},
    }
    if a.report:
        rep = {"line": line, "steps": [{"batch": st["batch"],
                                        "fractions": {str(f): [r.summary() for r in st["res"][f]] for f in FRACTIONS},
                                        "cross_eval": {k: np.asarray(v).tolist() for k, v in st["cross"].items()}}
                                       for st in steps]}
        with open(a.report, "w") as fh:
            json.dump(rep, fh, indent=1)
    if not a.no_cpu_baseline:
        log("timing the oracle on the host")
        line["cpu_baseline"] = cpu_baseline(cfg, launches_per_candidate(cfg, len(layers), len(FRACTIONS), SLICE))
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
