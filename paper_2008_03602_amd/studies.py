"""Studies built on the tuning path: TSI scaling and measurement isolation.

* TSI scaling (section 3.1.1 and Fig. 7a: one client's candidates spread over
  1, 2 and 4 tuning server instances). One layer's candidate list is screened
  on k disjoint CU slots at once; the k screening results are merged, the
  global top T re-measured on slot 0 and the winner selected with the usual
  tie rule. Per-layer tuning time is reported against k, and each winner is
  compared with the one a single slot finds.
* Isolation (section 2.2: a fixed GPU share is what lets concurrent tuning
  record the right latency). Fixed schedules are timed on slot 0 of the 25 %
  share alone, then while slots 1-3 run (i) the same kernels or (ii) an HBM
  copy, and on an unmasked stream while slots 1-3 run the same kernels (the
  analogue of sharing the GPU without a fixed share). Reported: latency
  inflation and whether the fastest of the schedules changes.
* Guided search (section 2.1, stage 4, and early stopping): per layer, the
  random-sample tuner and the annealing search with the same budget on the
  same slot; reported: candidates each needs before its best screened
  latency is within x of the random tuner's winner, both winners re-timed
  side by side, and where the patience rule stops the guided search.

Every slot has one host thread that runs the library calls for that slot (a
call releases the interpreter lock), so each slot keeps its own CU-masked
stream for the whole study.

Usage: python -m paper_2008_03602_amd.studies {tsi|isolation|search} [--layers N] [--candidates N] [--out F]
"""
from __future__ import annotations

import argparse
import json
import queue
import threading
import time
from concurrent.futures import Future
from typing import Callable, Dict, List, Sequence

import numpy as np
import torch

from . import _lib as L
from . import tuner as T
from . import workloads as W


class Slots:
    """One worker thread per CU slot; work for slot j runs on thread j."""

    def __init__(self, k: int):
        self.q: List[queue.Queue] = [queue.Queue() for _ in range(k)]
        self.threads = [threading.Thread(target=self._run, args=(j,), daemon=True) for j in range(k)]
        for t in self.threads:
            t.start()

    def _run(self, j: int) -> None:
        while True:
            item = self.q[j].get()
            if item is None:
                return
            fn, fut = item
            try:
                fut.set_result(fn())
            except BaseException as e:  # handed to the caller through the future
                fut.set_exception(e)

    def submit(self, j: int, fn: Callable) -> Future:
        fut: Future = Future()
        self.q[j].put((fn, fut))
        return fut

    def close(self) -> None:
        for q in self.q:
            q.put(None)
        for t in self.threads:
            t.join()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
        return False


def split_screen(ld: T.LayerData, cands: List[L.ct_schedule], cfg: W.TuneConfig, fraction: float, k: int,
                 slots: "Slots", ys: Sequence[torch.Tensor], y_ref=None) -> dict:
    """One client over k CU slots (ct_tune_split runs the k screens at once,
    the merge, the re-measure on slot 0 and the selection). Runs on slot 0's
    thread so that the study's threads stay one per slot."""
    r = slots.submit(0, lambda: T.tune_split(ld, cands, cfg, fraction, k, ys, y_ref=y_ref)).result()
    r.pop("result")
    return r


def tsi_scaling(layers: Sequence[T.LayerData], cands: Dict[int, List[L.ct_schedule]], cfg: W.TuneConfig,
                fraction: float = 0.25, ks: Sequence[int] = (1, 2, 4), verify_refs=None) -> dict:
    """Per layer and k: tuning time with the candidate list spread over k
    slots of `fraction`. Where a winner differs from the k = 1 winner, the two
    are re-timed side by side on slot 0 and their relative gap reported.
    verify_refs (optional, per layer id): fp32 device references that every
    screened candidate of every slot is checked against."""
    kmax = max(ks)
    out = {"fraction": fraction, "ks": list(ks), "layers": []}
    with Slots(kmax) as slots:
        ys = {ld.layer_id: [ld.y] + [torch.empty_like(ld.y) for _ in range(kmax - 1)] for ld in layers}
        # untimed pass: every slot's stream exists and every kernel has run once
        warm = L.make_opts(0, 1, 1, 16)
        for ld in layers:
            c = cands[ld.layer_id]
            futs = [slots.submit(j, lambda j=j, ld=ld, c=c: L.measure_candidates_mask(
                ld.op, c[j::kmax], L.ct_cu_mask(fraction, j), warm, ld.x, ld.w, ys[ld.layer_id][j]))
                for j in range(kmax)]
            for f in futs:
                f.result()
        for ld in layers:
            c = cands[ld.layer_id]
            row = {"layer": ld.op.name, "candidates": len(c), "runs": []}
            base = None
            for k in ks:
                r = split_screen(ld, c, cfg, fraction, k, slots, ys[ld.layer_id],
                                 (verify_refs or {}).get(ld.layer_id))
                if base is None:
                    base = r
                elif r["winner_pos"] != base["winner_pos"] and r["winner_pos"] >= 0 and base["winner_pos"] >= 0:
                    pair = [c[base["winner_pos"]], c[r["winner_pos"]]]
                    lat, st = slots.submit(0, lambda pair=pair: L.measure_candidates_mask(
                        ld.op, pair, L.ct_cu_mask(fraction, 0),
                        L.opts_from_protocol(cfg.stage2, batch=2, interleave=1), ld.x, ld.w, ld.y)).result()
                    r["flip_gap"] = float(abs(lat[0] - lat[1]) / min(lat[0], lat[1]))
                row["runs"].append(r)
            out["layers"].append(row)
            print("tsi %-7s %s" % (row["layer"], "  ".join(
                "k=%d %.2fs pos %d%s" % (r["k"], r["total_s"], r["winner_pos"],
                                         (" gap %.1f%%" % (100 * r["flip_gap"])) if "flip_gap" in r else "")
                for r in row["runs"])), flush=True)
    t = {k: sum(row["runs"][i]["total_s"] for row in out["layers"]) for i, k in enumerate(ks)}
    out["total_s"] = {str(k): v for k, v in t.items()}
    out["speedup"] = {str(k): t[ks[0]] / v for k, v in t.items()}
    flips = [r for row in out["layers"] for r in row["runs"][1:] if r["winner_pos"] != row["runs"][0]["winner_pos"]]
    out["winner_flips"] = len(flips)
    out["max_flip_gap"] = max([r.get("flip_gap", 0.0) for r in flips], default=0.0)
    return out


def isolation(ld: T.LayerData, scheds: List[L.ct_schedule], cfg: W.TuneConfig, slots: Slots,
              copy_bufs: Sequence, ys: Sequence[torch.Tensor], y_ref=None) -> dict:
    """Stage-2 latencies of fixed schedules on slot 0 of the 25 % share alone,
    with slots 1-3 running the same kernels, with slots 1-3 copying, and on
    an unmasked stream alone and with slots 1-3 running the same kernels.
    y_ref (optional): fp32 device reference that every timed schedule's output
    is checked against in every condition (statuses in "status")."""
    o = L.opts_from_protocol(cfg.stage2, batch=len(scheds), interleave=1)
    bg_opts = L.make_opts(0, 1, 10, len(scheds))
    copy_opts = L.make_opts(0, 1, 1, 1)
    statuses = {}

    def timed(mask, key):
        lat, st = slots.submit(0, lambda: L.measure_candidates_mask(ld.op, scheds, mask, o, ld.x, ld.w, ys[0],
                                                                    y_ref=y_ref, tol=1e-4)).result()
        statuses[key] = st.tolist()
        return np.where(st == L.S_OK, lat, np.inf).astype(np.float64)

    def with_load(kind: str, mask, key: str) -> np.ndarray:
        stop = threading.Event()

        def loop(j: int):
            m = L.ct_cu_mask(0.25, j)
            n = 0
            while not stop.is_set() or n == 0:
                if kind == "same":
                    L.measure_candidates_mask(ld.op, scheds, m, bg_opts, ld.x, ld.w, ys[j])
                else:
                    src, dst = copy_bufs[j - 1]
                    L.ct_probe_copy(m, src, dst, src.numel() * 4, copy_opts)
                n += 1
            return n

        futs = [slots.submit(j, lambda j=j: loop(j)) for j in (1, 2, 3)]
        time.sleep(0.05)  # the load is running before the timing starts
        try:
            return timed(mask, key)
        finally:
            stop.set()
            for f in futs:
                f.result()

    mask0 = L.ct_cu_mask(0.25, 0)
    full = L.ct_cu_mask(1.0, 0)
    res = {"layer": ld.op.name, "schedules": [T.describe_schedule(ld.op, s)["knobs"] for s in scheds]}
    lat = {"alone": timed(mask0, "alone"),
           "neighbours_same_kernels": with_load("same", mask0, "neighbours_same_kernels"),
           "neighbours_copying": with_load("copy", mask0, "neighbours_copying"),
           "unmasked_alone": timed(full, "unmasked_alone"),
           "unmasked_shared": with_load("same", full, "unmasked_shared")}
    res["latency_us"] = {k: v.tolist() for k, v in lat.items()}
    res["status"] = statuses
    res["inflation"] = {
        "neighbours_same_kernels": (lat["neighbours_same_kernels"] / lat["alone"]).tolist(),
        "neighbours_copying": (lat["neighbours_copying"] / lat["alone"]).tolist(),
        "unmasked_shared": (lat["unmasked_shared"] / lat["unmasked_alone"]).tolist()}
    res["fastest"] = {k: int(np.argmin(v)) for k, v in lat.items()}
    res["winner_flip"] = {k: res["fastest"][k] != res["fastest"][ref] for k, ref in
                          (("neighbours_same_kernels", "alone"), ("neighbours_copying", "alone"),
                           ("unmasked_shared", "unmasked_alone"))}
    return res


def isolation_study(layers: Sequence[T.LayerData], cands: Dict[int, List[L.ct_schedule]], cfg: W.TuneConfig,
                    n_sched: int = 8, copy_mib: int = 256) -> dict:
    """isolation() on each layer's n_sched best screened candidates at 25 %."""
    n = copy_mib * (1 << 18)
    copy_bufs = [(torch.ones(n, device="cuda:0"), torch.empty(n, device="cuda:0")) for _ in range(3)]
    out = {"layers": []}
    with Slots(4) as slots:
        for ld in layers:
            ys = [ld.y] + [torch.empty_like(ld.y) for _ in range(3)]
            lat, st = slots.submit(0, lambda: L.measure_candidates_mask(
                ld.op, cands[ld.layer_id], L.ct_cu_mask(0.25, 0), L.opts_from_protocol(cfg.stage1),
                ld.x, ld.w, ys[0])).result()
            top = L.ct_top_t(lat, st, n_sched)
            r = isolation(ld, [cands[ld.layer_id][i] for i in top], cfg, slots, copy_bufs, ys)
            out["layers"].append(r)
            inf = r["inflation"]
            print("isolation %-7s median (max) inflation: same kernels %.3f (%.3f), copying %.3f (%.3f), "
                  "unmasked shared %.3f (%.3f); fastest changes: %s" % (
                      ld.op.name, np.median(inf["neighbours_same_kernels"]), np.max(inf["neighbours_same_kernels"]),
                      np.median(inf["neighbours_copying"]), np.max(inf["neighbours_copying"]),
                      np.median(inf["unmasked_shared"]), np.max(inf["unmasked_shared"]),
                      json.dumps(r["winner_flip"])), flush=True)
    for key in ("neighbours_same_kernels", "neighbours_copying", "unmasked_shared"):
        v = np.concatenate([r["inflation"][key] for r in out["layers"]])
        out[key] = {"median_inflation": float(np.median(v)), "max_inflation": float(np.max(v)),
                    "flips": int(sum(r["winner_flip"][key] for r in out["layers"]))}
    return out


def first_within(lat: np.ndarray, target: float) -> int:
    """1-based count of candidates screened before the running best is at or
    below target (-1 if never)."""
    best = np.minimum.accumulate(np.where(np.isfinite(lat), lat, np.inf))
    hit = np.nonzero(best <= target)[0]
    return int(hit[0]) + 1 if len(hit) else -1


def search_study(layers: Sequence[T.LayerData], cands: Dict[int, List[L.ct_schedule]], cfg: W.TuneConfig,
                 fraction: float = 0.25, within: float = 0.05, patience: int = 48, seed: int = 0) -> dict:
    """Random-sample tuning against guided search with the same budget (the
    sample size), on slot 0 of `fraction`, layer by layer."""
    mask = L.ct_cu_mask(fraction, 0)
    o1 = L.opts_from_protocol(cfg.stage1)
    o2 = L.opts_from_protocol(cfg.stage2, batch=cfg.top_t, interleave=1)
    out = {"fraction": fraction, "within": within, "patience": patience, "layers": []}
    for ld in layers:
        c = cands[ld.layer_id]
        rnd = T.tune_clients([[ld]], [mask], cands, cfg, fraction)[0]
        target = (1.0 + within) * rnd.winner_lat_us
        so = L.make_search_opts(seed=seed, batch=16, budget=len(c), patience=0, eps=cfg.eps)
        g_meas, g_lat, g_st, g_res = L.ct_search(ld.op, so, mask, o1, o2, cfg.top_t, cfg.eps, ld.x, ld.w, ld.y)
        so_es = L.make_search_opts(seed=seed, batch=16, budget=len(c), patience=patience, eps=cfg.eps)
        e_meas, e_lat, e_st, e_res = L.ct_search(ld.op, so_es, mask, o1, o2, cfg.top_t, cfg.eps, ld.x, ld.w, ld.y)
        # the three winners side by side, repeats interleaved
        trio = [rnd.winner, g_meas[g_res["winner"]], e_meas[e_res["winner"]]]
        lat, st = L.measure_candidates_mask(ld.op, trio, mask, L.opts_from_protocol(cfg.stage2, batch=3, interleave=1),
                                            ld.x, ld.w, ld.y)
        r1 = np.where(rnd.status1 == L.S_OK, rnd.lat1, np.inf)
        row = {"layer": ld.op.name, "budget": len(c),
               "random_winner_us": float(lat[0]), "guided_winner_us": float(lat[1]),
               "early_stop_winner_us": float(lat[2]),
               "random_to_within": first_within(r1, target),
               "guided_to_within": first_within(np.where(g_st == L.S_OK, g_lat, np.inf), target),
               "early_stop_measured": e_res["n_measured"], "early_stopped": bool(e_res["stopped_early"]),
               "guided_propose_s": g_res["propose_s"], "guided_measure_s": g_res["measure_s"],
               "guided_frac_of_scaled_peak": ld.op.flops() / (float(lat[1]) * 1e-6) / 1e12 /
                                             (T.PEAK_FP32_TFLOPS * fraction),
               "guided_families": {str(f): int(sum(1 for s in g_meas if s.family == f)) for f in (1, 2, 3, 4)},
               "random_families": {str(f): int(sum(1 for s in c if s.family == f)) for f in (1, 2, 3, 4)}}
        out["layers"].append(row)
        print("search %-7s winners (us) random %.2f guided %.2f (%.1f%% of the scaled peak) early-stop %.2f "
              "(%d measured%s); to within %d%%: random %d, guided %d; propose %.2fs measure %.2fs" % (
                  row["layer"], lat[0], lat[1], 100 * row["guided_frac_of_scaled_peak"], lat[2],
                  row["early_stop_measured"],
                  ", stopped" if row["early_stopped"] else "", round(100 * within), row["random_to_within"],
                  row["guided_to_within"], row["guided_propose_s"], row["guided_measure_s"]), flush=True)
    rows = out["layers"]
    out["guided_vs_random_winner"] = float(np.exp(np.mean([np.log(r["guided_winner_us"] / r["random_winner_us"])
                                                            for r in rows])))
    out["early_stop_vs_random_winner"] = float(np.exp(np.mean([np.log(r["early_stop_winner_us"] /
                                                                      r["random_winner_us"]) for r in rows])))
    out["early_stop_budget_share"] = float(np.mean([r["early_stop_measured"] / r["budget"] for r in rows]))
    g = [r["guided_to_within"] for r in rows]
    rr = [r["random_to_within"] for r in rows]
    out["guided_reached"] = int(sum(v > 0 for v in g))
    out["random_reached"] = int(sum(v > 0 for v in rr))
    out["median_guided_to_within"] = float(np.median([v if v > 0 else np.inf for v in g]))
    out["median_random_to_within"] = float(np.median([v if v > 0 else np.inf for v in rr]))
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description="TSI scaling and isolation studies on the ResNet-18 layers")
    ap.add_argument("study", choices=("tsi", "isolation", "search"))
    ap.add_argument("--layers", type=int, default=12, help="first N ResNet-18 layers")
    ap.add_argument("--candidates", type=int, default=128)
    ap.add_argument("--fraction", type=float, default=0.25, help="CU share of the search study")
    ap.add_argument("--only", default=None, help="comma-separated layer names (default: the first N)")
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    L.ct_init(0)
    cfg = W.config(2)
    cfg.n_candidates = a.candidates
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops[:a.layers])]
    if a.only:
        layers = [ld for ld in layers if ld.op.name in a.only.split(",")]
    cands = T.sample_all(layers, cfg)
    if a.study == "tsi":
        rep = tsi_scaling(layers, cands, cfg)
        print("tsi total seconds by k:", json.dumps(rep["total_s"]), "speedup:", json.dumps(rep["speedup"]),
              "winner flips:", rep["winner_flips"], "max gap %.3f" % rep["max_flip_gap"], flush=True)
    elif a.study == "search":
        rep = search_study(layers, cands, cfg, fraction=a.fraction)
        print("search summary:", json.dumps({k: v for k, v in rep.items() if k != "layers"}), flush=True)
    else:
        rep = isolation_study(layers, cands, cfg)
        print("isolation summary:", json.dumps({k: rep[k] for k in
                                                ("neighbours_same_kernels", "neighbours_copying", "unmasked_shared")}),
              flush=True)
    if a.out:
        with open(a.out, "w") as fh:
            json.dump(rep, fh, indent=1)
    L.ct_shutdown()
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
