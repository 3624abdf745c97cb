"""Tuning runs over the C ABI: clients on CU slots, selection, cross-evaluation.

This module only prepares inputs and marshals arguments; sampling, timing,
selection and the client threads all run inside libconvtune.

The paper's loop (section 2.1): select candidates (random with no history),
build, profile on the device, pick the best. Its scaling (section 3.1.1):
several profiling servers with fixed GPU shares, and a model's operators
sharded over several tuning clients whose results are merged. Here a client
is a library thread with its own CU-masked stream; the operators of a model
are taken by the clients from one shared queue, largest first (or dealt
round-robin), and the merged result is the per-layer winner. Cross-evaluation (section 2.2.1, Tables 1-2) re-runs the schedule
tuned at one share on every other share.
"""
from __future__ import annotations

import ctypes
import json
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import _lib as L
from . import synth
from . import workloads as W

PEAK_FP32_TFLOPS = 157.3      # MI355X vector / matrix fp32, 256 CUs at 2.4 GHz
PEAK_BF16_TFLOPS = 2516.6     # dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0

# Concurrent clients per CU share. The device deals hardware queues to 4
# dispatch pipes in creation order, and the library creates a share's slot
# streams one after another, so slots j and j + 4 of a share land on one pipe.
# Measured at 12.5 % (8 slots of 32 CUs): the one neighbour on slot 0's pipe
# inflates slot 0's latencies 1.8-2.5x, the six on other pipes 1.06-1.10x
# together. So a share runs at most 4 clients (one per pipe), on slots 0-3.
MAX_CLIENTS = 4


@dataclass
class LayerData:
    """Device buffers of one layer: seeded synthetic x and w, an output y."""
    op: W.Op
    layer_id: int
    x: torch.Tensor
    w: torch.Tensor
    y: torch.Tensor


def make_layer(op: W.Op, cfg: W.TuneConfig, layer_id: int, device: str = "cuda:0") -> LayerData:
    bf16 = op.dtype == W.DT_BF16
    x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), cfg.dist, cfg.seed, cfg.config_id, layer_id, bf16=bf16)
    if bf16:
        xd = torch.from_numpy(synth.bf16_bits(x).view(np.int16).copy()).to(device)
        wd = torch.from_numpy(synth.bf16_bits(w).view(np.int16).copy()).to(device)
    else:
        xd = torch.from_numpy(x).to(device)
        wd = torch.from_numpy(w).to(device)
    yd = torch.empty(op.y_shape(), dtype=torch.float32, device=device)
    return LayerData(op, layer_id, xd, wd, yd)


@dataclass
class JobResult:
    op: W.Op
    layer_id: int
    client: int
    fraction: float
    candidates: List[L.ct_schedule]
    lat1: np.ndarray
    status1: np.ndarray
    top_pos: np.ndarray
    lat2: np.ndarray
    winner_pos: int
    winner_lat_us: float
    t_start: float
    t_end: float

    @property
    def winner(self) -> Optional[L.ct_schedule]:
        return self.candidates[self.winner_pos] if self.winner_pos >= 0 else None

    def summary(self) -> dict:
        s = self.winner
        d = {"layer": self.op.name, "client": self.client, "fraction": self.fraction,
             "n_candidates": len(self.candidates),
             "n_ok": int(np.sum(self.status1 == L.S_OK)),
             "status_counts": {L.STATUS_NAMES[k]: int(np.sum(self.status1 == k)) for k in L.STATUS_NAMES
                               if np.any(self.status1 == k)},
             "winner_pos": self.winner_pos, "winner_lat_us": self.winner_lat_us,
             "t_start": self.t_start, "t_end": self.t_end}
        d["top"] = [{"pos": int(p), "lat2_us": float(l), "family": int(self.candidates[int(p)].family),
                     "knobs": list(describe_schedule(self.op, self.candidates[int(p)])["knobs"].values())}
                    for p, l in zip(self.top_pos, self.lat2)]
        if s is not None:
            d["winner"] = describe_schedule(self.op, s)
            d["winner_tflops"] = self.op.flops() / (self.winner_lat_us * 1e-6) / 1e12
            d["winner_gbps"] = self.op.bytes_moved() / (self.winner_lat_us * 1e-6) / 1e9
        return d


def describe_schedule(op: W.Op, s: L.ct_schedule) -> dict:
    nk, _ = L.ct_grid_info(s.family)
    names = {1: ["toh", "tow", "tk", "mk", "mw", "lds", "ct", "split", "unroll"],
             2: ["tc", "toh", "tow", "vec", "rpt", "lds", "nb", "order", "q4"],
             3: ["mfma", "tm", "tn", "wm", "wn", "kc", "lds", "split", "swizzle"],
             4: ["mfma", "tm", "tn", "wm", "wn", "ws", "tpw", "cpc", "stages", "split"]}[s.family]
    d = {"family": W.FAMILY_NAMES[s.family], "knobs": {names[i]: int(s.knob[i]) for i in range(nk)},
         "grid_index": L.ct_grid_encode(s)}
    d.update(L.ct_launch_shape(op, s))
    return d


class _Keep:
    """Holds numpy/ctypes buffers alive for the duration of a library call."""

    def __init__(self):
        self.items = []

    def add(self, x):
        self.items.append(x)
        return x


def fill_job(jb, op: W.Op, layer_id: int, x, w, y, c: List[L.ct_schedule], top_t: int, keep: _Keep,
             y_ref: Optional[torch.Tensor] = None, verify_tol: float = 1e-4, recorded: Optional[dict] = None):
    """Point one ct_tune_job at a layer's buffers, candidates and result arrays.
    recorded (resume): {sample position: (lat_us, status)} of candidates that a
    log already holds; they are passed as skipped, with their recorded values."""
    arr = keep.add(L.schedule_array(c))
    n = len(c)
    lat1 = keep.add(np.zeros(max(n, 1), np.float32))
    st1 = keep.add(np.zeros(max(n, 1), np.int32))
    top = keep.add(np.zeros(top_t, np.int32))
    lat2 = keep.add(np.zeros(top_t, np.float32))
    jb.op = L.make_op(op)
    jb.x, jb.w, jb.y = L._ptr(x), L._ptr(w), L._ptr(y)
    jb.cands, jb.n_cands = arr, n
    jb.layer_id = layer_id
    if y_ref is not None:
        jb.verify = L.ct_verify(y_ref.data_ptr(), verify_tol)
    if recorded:
        skip = keep.add(np.zeros(max(n, 1), np.uint8))
        for pos, (lat, st) in recorded.items():
            if 0 <= pos < n:
                skip[pos] = 1
                lat1[pos] = np.float32(lat)
                st1[pos] = st
        jb.skip = skip.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8))
    jb.lat1_us = lat1.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    jb.status1 = st1.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    jb.top_t = top_t
    jb.top_pos = top.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    jb.lat2_us = lat2.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    return (c, lat1, st1, top, lat2)


def _fill_job(jb, ld: LayerData, c: List[L.ct_schedule], cfg: W.TuneConfig, keep: _Keep,
              verify_refs: Optional[Dict[int, torch.Tensor]], verify_tol: float, recorded=None):
    ref = verify_refs.get(ld.layer_id) if verify_refs is not None else None
    return (ld,) + fill_job(jb, ld.op, ld.layer_id, ld.x, ld.w, ld.y, c, cfg.top_t, keep, ref, verify_tol,
                            recorded)


def _result(jb, meta, client: int, fraction: float) -> JobResult:
    ld, c, lat1, st1, top, lat2 = meta
    n, nt = len(c), jb.n_top
    return JobResult(ld.op, ld.layer_id, client, fraction, list(c), lat1[:n].copy(), st1[:n].copy(),
                     top[:nt].copy(), lat2[:nt].copy(), jb.winner_pos, jb.winner_lat_us, jb.t_start_s, jb.t_end_s)


def _clients(masks: Sequence[np.ndarray], pin_cores: bool, log_paths: Optional[Sequence[str]] = None,
             keep: Optional[_Keep] = None) -> ctypes.Array:
    clients = (L.ct_client * len(masks))()
    for j, m in enumerate(masks):
        for k, v in enumerate(m):
            clients[j].cu_mask[k] = int(v)
        clients[j].host_core = j if pin_cores else -1
        if log_paths is not None:
            b = log_paths[j].encode()
            if keep is not None:
                keep.add(b)
            clients[j].log_path = b
    return clients


@dataclass
class ClientStats:
    """What the library reports per client after a run."""
    n_measured: int
    t_start: float
    t_end: float
    cands_per_s: float


def client_stats(clients: ctypes.Array) -> List[ClientStats]:
    return [ClientStats(int(c.n_measured), c.t_start_s, c.t_end_s, c.cands_per_s) for c in clients]


def tune_clients(assignments: Sequence[Sequence[LayerData]], masks: Sequence[np.ndarray],
                 cands: Dict[int, List[L.ct_schedule]], cfg: W.TuneConfig, fraction: float,
                 verify_refs: Optional[Dict[int, torch.Tensor]] = None, verify_tol: float = 1e-4,
                 pin_cores: bool = True, batch: int = 16) -> List[JobResult]:
    """Run one client per assignment, concurrently, each on its CU mask.

    assignments[j] lists the layers of client j; cands[layer_id] is that
    layer's candidate list (sample order). Returns one JobResult per layer.
    """
    keep = _Keep()
    clients = _clients(masks, pin_cores)
    jobs_meta = []
    for j, layers in enumerate(assignments):
        jobs = keep.add((L.ct_tune_job * max(len(layers), 1))())
        for i, ld in enumerate(layers):
            jobs_meta.append((j, i, _fill_job(jobs[i], ld, cands[ld.layer_id], cfg, keep, verify_refs, verify_tol)))
        clients[j].jobs = ctypes.cast(jobs, ctypes.POINTER(L.ct_tune_job))
        clients[j].n_jobs = len(layers)
    o1 = L.opts_from_protocol(cfg.stage1, batch=batch)
    o2 = L.opts_from_protocol(cfg.stage2, batch=cfg.top_t, interleave=1)
    L.ct_tune_clients(clients, o1, o2, cfg.eps)
    out = []
    for (j, i, meta) in jobs_meta:
        jb = ctypes.cast(clients[j].jobs, ctypes.POINTER(L.ct_tune_job))[i]
        out.append(_result(jb, meta, j, fraction))
    return out


class SharedRun(list):
    """JobResults of one shared-queue run, plus the library's client figures."""
    clients: List[ClientStats]
    cands_per_s: float


def tune_shared(layers: Sequence[LayerData], masks: Sequence[np.ndarray], cands: Dict[int, List[L.ct_schedule]],
                cfg: W.TuneConfig, fraction: float, verify_refs: Optional[Dict[int, torch.Tensor]] = None,
                verify_tol: float = 1e-4, pin_cores: bool = True, batch: int = 16,
                log_paths: Optional[Sequence[str]] = None,
                recorded: Optional[Dict[int, dict]] = None) -> "SharedRun":
    """Run one client per mask on a shared queue of layers, taken in the given
    order by whichever client is idle first. Returns one JobResult per layer
    (a SharedRun, which also carries the per-client and aggregate candidates/s
    that the library computed). log_paths: one JSON-lines log per client;
    recorded (resume): per layer id, the candidates a log already holds."""
    keep = _Keep()
    clients = _clients(masks, pin_cores, log_paths, keep)
    jobs = (L.ct_tune_job * max(len(layers), 1))()
    metas = [_fill_job(jobs[i], ld, cands[ld.layer_id], cfg, keep, verify_refs, verify_tol,
                       (recorded or {}).get(ld.layer_id))
             for i, ld in enumerate(layers)]
    o1 = L.opts_from_protocol(cfg.stage1, batch=batch)
    o2 = L.opts_from_protocol(cfg.stage2, batch=cfg.top_t, interleave=1)
    owner = L.ct_tune_shared(clients, (L.ct_tune_job * len(layers)).from_address(ctypes.addressof(jobs)),
                             o1, o2, cfg.eps)
    out = SharedRun(_result(jobs[i], metas[i], int(owner[i]), fraction) for i in range(len(layers)))
    out.clients = client_stats(clients)
    out.cands_per_s = L.ct_throughput(clients)
    return out


def tune_split(ld: LayerData, c: List[L.ct_schedule], cfg: W.TuneConfig, fraction: float, k: int,
               ys: Sequence[torch.Tensor], y_ref: Optional[torch.Tensor] = None,
               verify_tol: float = 1e-4) -> dict:
    """One client over k CU slots (ct_tune_split): the layer's candidates are
    screened on slots 0..k-1 of `fraction` at once, then re-measured and
    selected on slot 0. ys: k output buffers."""
    keep = _Keep()
    jb = L.ct_tune_job()
    meta = (ld,) + fill_job(jb, ld.op, ld.layer_id, ld.x, ld.w, ys[0], c, cfg.top_t, keep, y_ref, verify_tol)
    masks = [L.ct_cu_mask(fraction, j) for j in range(k)]
    t0 = time.perf_counter()
    screen_s = L.ct_tune_split(jb, masks, ys[:k], L.opts_from_protocol(cfg.stage1),
                               L.opts_from_protocol(cfg.stage2, batch=cfg.top_t, interleave=1), cfg.eps)
    total_s = time.perf_counter() - t0
    r = _result(jb, meta, 0, fraction)
    return {"k": k, "screen_s": screen_s, "total_s": total_s, "screened_ok": int(np.sum(r.status1 == L.S_OK)),
            "status_counts": {L.STATUS_NAMES[s]: int(np.sum(r.status1 == s)) for s in L.STATUS_NAMES
                              if np.any(r.status1 == s)},
            "winner_pos": r.winner_pos, "winner_lat_us": r.winner_lat_us, "result": r}


def largest_first(layers: Sequence[LayerData]) -> List[LayerData]:
    """Queue order for a shared queue: layers by decreasing FLOPs (ties in table order)."""
    return sorted(layers, key=lambda ld: (-ld.op.flops(), ld.layer_id))


def round_robin(layers: Sequence[LayerData], k: int) -> List[List[LayerData]]:
    """Shard a model's layers over k clients in table order (layer i -> client i mod k)."""
    return [[ld for i, ld in enumerate(layers) if i % k == j] for j in range(k)]


def cross_eval(ld: LayerData, winners: Sequence[L.ct_schedule], masks: Sequence[np.ndarray],
               proto: W.Protocol, batch: int = 8) -> np.ndarray:
    """M[i][j]: latency (us) of winners[i] on masks[j], repeats interleaved."""
    o = L.opts_from_protocol(proto, batch=batch, interleave=1)
    return L.ct_cross_eval(ld.op, winners, masks, o, ld.x, ld.w, ld.y)


def throughput(n_candidates: int, t_first_start: float, t_last_end: float) -> float:
    """Candidates per second over the makespan (first start to last end)."""
    span = t_last_end - t_first_start
    return n_candidates / span if span > 0 else float("nan")


def sample_all(layers: Sequence[LayerData], cfg: W.TuneConfig, uniform: bool = False) -> Dict[int, List[L.ct_schedule]]:
    """Each layer's seeded candidate list: equal shares per kernel family
    (ct_sample), or one shuffle of the whole valid space (ct_sample_uniform)."""
    f = L.ct_sample_uniform if uniform else L.ct_sample
    return {ld.layer_id: f(ld.op, cfg.seed, cfg.config_id, ld.layer_id, cfg.n_candidates) for ld in layers}


def tune_model_at_fraction(layers: Sequence[LayerData], cands, cfg: W.TuneConfig, fraction: float,
                           clients: Optional[int] = None, sharding: str = "queue", **kw) -> List[JobResult]:
    """Tune every layer at CU share `fraction`, with as many concurrent clients as
    disjoint slots of that share fit on the device (or `clients`).

    sharding "queue": the clients take layers from one queue, largest first;
    "round_robin": layer i goes to client i mod k, in table order."""
    k = clients or min(MAX_CLIENTS, max(1, int(round(1.0 / fraction))))
    k = min(k, len(layers))
    masks = [L.ct_cu_mask(fraction, j) for j in range(k)]
    if sharding == "queue":
        res = tune_shared(largest_first(layers), masks, cands, cfg, fraction, **kw)
        res.sort(key=lambda r: r.layer_id)
        return res
    if sharding != "round_robin":
        raise ValueError("sharding is 'queue' or 'round_robin'")
    return tune_clients(round_robin(layers, k), masks, cands, cfg, fraction, **kw)


def fraction_report(results: Sequence[JobResult]) -> dict:
    """Candidates, makespan and candidates/s of one share's run. For a shared
    queue run the figures are the library's (per client and aggregate)."""
    t0 = min(r.t_start for r in results)
    t1 = max(r.t_end for r in results)
    n = sum(len(r.candidates) for r in results)
    rep = {"candidates": n, "seconds": t1 - t0, "candidates_per_s": throughput(n, t0, t1),
           "clients": len({r.client for r in results})}
    if isinstance(results, SharedRun):
        rep["candidates_per_s"] = results.cands_per_s
        rep["seconds"] = max(c.t_end for c in results.clients) - min(c.t_start for c in results.clients)
        rep["per_client_candidates_per_s"] = [c.cands_per_s for c in results.clients]
    return rep


def read_logs(paths: Sequence[str]) -> dict:
    """Merge per-client JSON-lines logs (append-only; a cut last line is
    skipped): {"cands": {layer: {pos: (lat_us, status, family, knobs)}},
    "jobs": {layer: record of the job's end}}. A candidate recorded twice keeps
    its first record and is counted in "duplicates"."""
    cands: Dict[int, dict] = {}
    jobs: Dict[int, dict] = {}
    dup = 0
    for p in paths:
        try:
            fh = open(p)
        except FileNotFoundError:
            continue
        with fh:
            for line in fh:
                try:
                    rec = json.loads(line)
                except ValueError:
                    continue
                if rec.get("kind") == "cand":
                    d = cands.setdefault(int(rec["layer"]), {})
                    pos = int(rec["pos"])
                    if pos in d:
                        dup += 1
                        continue
                    lat = rec["lat_us"]
                    d[pos] = (float("inf") if lat is None else float(lat), int(rec["status"]), int(rec["family"]),
                              list(rec["knobs"]))
                elif rec.get("kind") == "job" and int(rec.get("rc", 0)) == 0:
                    jobs[int(rec["layer"])] = rec
    return {"cands": cands, "jobs": jobs, "duplicates": dup}


def resume_state(logs: dict, cands: Dict[int, List[L.ct_schedule]]) -> Dict[int, dict]:
    """Per layer id, {pos: (lat_us, status)} of recorded candidates, after
    checking that each recorded schedule is the one at that sample position."""
    out: Dict[int, dict] = {}
    for layer, recs in logs["cands"].items():
        c = cands.get(layer)
        if c is None:
            continue
        d = {}
        for pos, (lat, st, fam, knobs) in recs.items():
            s = c[pos] if pos < len(c) else None
            if s is None or int(s.family) != fam or [int(v) for v in s.knob[:len(knobs)]] != knobs:
                raise ValueError("log of layer %d does not match the candidate list at position %d" % (layer, pos))
            d[pos] = (lat, st)
        out[layer] = d
    return out


def cross_eval_regret(matrices: Dict[str, list], fractions: Sequence[float]) -> List[List[float]]:
    """Mean over layers of M[f][g] / min_f' M[f'][g]: how much slower the
    schedule tuned at share f runs at share g than the best of the winners."""
    n = len(fractions)
    acc = np.zeros((n, n))
    for M in matrices.values():
        M = np.asarray(M, dtype=np.float64)
        acc += M / M.min(axis=0, keepdims=True)
    return (acc / max(len(matrices), 1)).tolist()


def model_aggregates(matrices: Dict[str, list], fractions: Sequence[float]) -> dict:
    """Model-level view of the cross-evaluation (the paper's Tables 1-3).

    total[f][g] = sum over layers of multiplicity x M[f][g]: the model's conv
    time at share g when every layer runs the schedule tuned at share f.
    best[g] = the same with each layer's best winner for g. The sweet spot is
    the tuning share whose totals are closest to best on average over g."""
    n = len(fractions)
    total = np.zeros((n, n))
    best = np.zeros(n)
    for name, M in matrices.items():
        M = np.asarray(M, dtype=np.float64)
        k = W.multiplicity(name)
        total += k * M
        best += k * M.min(axis=0)
    ratio = total / best[None, :]
    mean = ratio.mean(axis=1)
    return {"total_us": total.tolist(), "best_us": best.tolist(), "ratio_to_best": ratio.tolist(),
            "mean_ratio_per_tuning_share": mean.tolist(), "sweet_spot": float(fractions[int(np.argmin(mean))])}


def determinism_report(runs: Sequence[dict], layers: Sequence[LayerData], cands, cfg: W.TuneConfig) -> dict:
    """Winners of repeated tunings with one seed: the candidate lists are
    identical by construction; a winner may differ only inside the tie band.
    Every (layer, share) whose winner changed is re-timed side by side (the
    stage-2 protocol) and its gap reported."""
    by_id = {ld.layer_id: ld for ld in layers}
    flips = []
    for key in runs[0]:
        seen = sorted({r[key] for r in runs if r[key] >= 0})
        if len(seen) <= 1:
            continue
        layer, f = key
        ld = by_id[layer]
        sched = [cands[layer][p] for p in seen]
        lat, st = L.measure_candidates_mask(ld.op, sched, L.ct_cu_mask(f, 0),
                                            L.opts_from_protocol(cfg.stage2, batch=len(sched), interleave=1),
                                            ld.x, ld.w, ld.y)
        lat = [float(v) for v in lat]
        flips.append({"layer": ld.op.name, "fraction": f, "positions": seen, "latency_us": lat,
                      "gap": (max(lat) - min(lat)) / min(lat)})
    n = len(runs[0])
    return {"reruns": len(runs), "cells": n, "flipped_cells": len(flips),
            "identical": n - len(flips), "max_gap": max([x["gap"] for x in flips], default=0.0), "flips": flips}


def find_layer(name: str):
    """(op, config, layer position) of a named layer of configurations 1-5."""
    for cid in range(1, 6):
        cfg = W.config(cid)
        for i, op in enumerate(cfg.ops):
            if op.name == name:
                return op, cfg, i
    raise KeyError("no layer named %r in configurations 1-5" % name)


def replay(layer: str, family: int, knobs: Sequence[int], fraction: float, launches: int,
           copy_mib: int) -> dict:
    """Run one schedule of one layer `launches` times back to back on slot 0 of
    `fraction`, then (if copy_mib > 0) the library's copy kernel over copy_mib
    MiB, so that a profiler run sees the kernel alone next to a transfer of
    known size."""
    op, cfg, i = find_layer(layer)
    ld = make_layer(op, cfg, i)
    s = L.make_schedule(family, list(knobs))
    if L.ct_validate(op, s) != 0:
        raise ValueError("invalid schedule: " + L.ct_last_error())
    mask = L.ct_cu_mask(fraction, 0)
    lat, st = L.measure_candidates_mask(op, [s], mask, L.make_opts(1, 1, launches, 1), ld.x, ld.w, ld.y)
    out = {"layer": layer, "kernel": L.ct_kernel_name(op, s), "schedule": describe_schedule(op, s),
           "fraction": fraction, "launches": launches, "status": int(st[0]), "latency_us": float(lat[0]),
           "tflops": op.flops() / (float(lat[0]) * 1e-6) / 1e12, "flops": op.flops(),
           "bytes_moved": op.bytes_moved(), "tbps": op.bytes_moved() / (float(lat[0]) * 1e-6) / 1e12,
           "dtype": "bf16" if op.dtype == W.DT_BF16 else "f32"}
    if copy_mib > 0:
        n = copy_mib * (1 << 20)
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        out["copy_bytes_each_way"] = n
        out["copy_gbps"] = L.ct_probe_copy(mask, src, dst, n, L.make_opts(1, 1, 1, 1))
    torch.cuda.synchronize()
    return out


def main(argv=None) -> int:
    import argparse
    ap = argparse.ArgumentParser(description="Run a tuning configuration (1-5) and write a JSON report, "
                                             "or replay one schedule (--replay).")
    ap.add_argument("--config", type=int, default=None)
    ap.add_argument("--out", default=None)
    ap.add_argument("--clients", type=int, default=None)
    ap.add_argument("--layers", type=int, default=None, help="only the first N layers")
    ap.add_argument("--candidates", type=int, default=None)
    ap.add_argument("--fractions", default=None, help="comma-separated CU shares (default: the config's)")
    ap.add_argument("--no-cross-eval", action="store_true", help="skip the cross-evaluation")
    ap.add_argument("--sharding", default="queue", choices=("queue", "round_robin"),
                    help="how a model's layers are spread over the clients")
    ap.add_argument("--replay", default=None, metavar="LAYER:FAMILY:K0,K1,...",
                    help="run one schedule of one layer and print its latency")
    ap.add_argument("--fraction", type=float, default=1.0, help="CU share for --replay")
    ap.add_argument("--launches", type=int, default=200, help="back-to-back launches for --replay")
    ap.add_argument("--copy-mib", type=int, default=0, help="--replay: also run the copy kernel over this many MiB")
    ap.add_argument("--uniform", action="store_true", help="sample the whole valid space uniformly (no family quotas)")
    ap.add_argument("--reruns", type=int, default=1,
                    help="run the tuning this many times with the same seed and report winner flips")
    a = ap.parse_args(argv)
    if a.replay:
        layer, fam, knobs = a.replay.split(":")
        L.ct_init(0)
        out = replay(layer, int(fam), [int(k) for k in knobs.split(",")], a.fraction, a.launches, a.copy_mib)
        print(json.dumps(out), flush=True)
        return 0 if out["status"] == L.S_OK else 1
    if a.config is None:
        ap.error("--config or --replay is required")
    cfg = W.config(a.config)
    if a.candidates:
        cfg.n_candidates = a.candidates
    if a.fractions:
        cfg.fractions = tuple(float(f) for f in a.fractions.split(","))
    ops = cfg.ops[:a.layers] if a.layers else cfg.ops
    L.ct_init(0)
    layers = [make_layer(op, cfg, i) for i, op in enumerate(ops)]
    cands = sample_all(layers, cfg, uniform=a.uniform)
    report = {"config": cfg.describe(), "sampler": "uniform" if a.uniform else "family quotas", "fractions": {}}
    winners = {}
    runs = []  # per rerun: {(layer, fraction): winner sample position}
    for rerun in range(max(1, a.reruns)):
        again = sample_all(layers, cfg, uniform=a.uniform)
        same = all([L.schedule_tuple(s) for s in again[k]] == [L.schedule_tuple(s) for s in cands[k]] for k in cands)
        if not same:
            raise RuntimeError("candidate lists differ between reruns of the same seed")
        pos = {}
        for f in cfg.fractions:
            res = tune_model_at_fraction(layers, cands, cfg, f, clients=a.clients, sharding=a.sharding)
            for r in res:
                pos[(r.layer_id, f)] = r.winner_pos
            if rerun:
                continue
            report["fractions"][str(f)] = {"throughput": fraction_report(res),
                                           "layers": [r.summary() for r in res]}
            for r in res:
                winners.setdefault(r.layer_id, {})[f] = r.winner
            print("fraction %.3f: %s" % (f, json.dumps(report["fractions"][str(f)]["throughput"])), flush=True)
        runs.append(pos)
        if rerun:
            print("rerun %d: %d of %d winners as in the first run" % (
                rerun, sum(pos[k] == runs[0][k] for k in pos), len(pos)), flush=True)
    if len(runs) > 1:
        report["determinism"] = determinism_report(runs, layers, cands, cfg)
        print("determinism:", json.dumps({k: v for k, v in report["determinism"].items() if k != "flips"}),
              flush=True)
    thr = {f: report["fractions"][str(f)]["throughput"]["candidates_per_s"] for f in cfg.fractions}
    if 1.0 in thr and len(thr) > 1:
        report["throughput_vs_one_full_gpu_client"] = {str(f): thr[f] / thr[1.0] for f in cfg.fractions}
        print("candidates/s relative to one full-GPU client:",
              json.dumps(report["throughput_vs_one_full_gpu_client"]), flush=True)
    if len(cfg.fractions) > 1 and not a.no_cross_eval:
        masks = [L.ct_cu_mask(f, 0) for f in cfg.fractions]
        report["cross_eval"] = {}
        for ld in layers:
            ws = [winners[ld.layer_id][f] for f in cfg.fractions]
            if any(s is None for s in ws):
                continue
            M = cross_eval(ld, ws, masks, cfg.stage2)
            report["cross_eval"][ld.op.name] = M.tolist()
            print("cross-eval %s done" % ld.op.name, flush=True)
        report["cross_eval_regret"] = cross_eval_regret(report["cross_eval"], cfg.fractions)
        print("cross-eval regret (rows: tuned at, columns: run at; mean over layers of "
              "latency / best latency in the column):", flush=True)
        for f, row in zip(cfg.fractions, report["cross_eval_regret"]):
            print("  %5.3f: %s" % (f, " ".join("%6.3f" % v for v in row)), flush=True)
        agg = model_aggregates(report["cross_eval"], cfg.fractions)
        report["model"] = agg
        print("model conv time / best, by tuning share (rows) and run share (columns):", flush=True)
        for f, row in zip(cfg.fractions, agg["ratio_to_best"]):
            print("  %5.3f: %s" % (f, " ".join("%6.3f" % v for v in row)), flush=True)
        print("sweet spot (lowest mean ratio): tuned at %.3f" % agg["sweet_spot"], flush=True)
    if a.out:
        with open(a.out, "w") as fh:
            json.dump(report, fh, indent=1)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
