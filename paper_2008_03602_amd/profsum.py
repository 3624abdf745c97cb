"""Summarise rocprofv3 output: per-kernel statistics, the bench's roofline
kernel, and HBM traffic from FETCH_SIZE / WRITE_SIZE counter runs.

Usage:
  python -m paper_2008_03602_amd.profsum --trace DIR [--bench FILE] [--replay FILE]
      [--fetch DIR --write DIR] [--out profiles/x.md] [--cmd "..."]...

--trace DIR   rocprofv3 --kernel-trace output: a rocpd database (``*.db``, the
              default format) or ``*kernel_trace.csv`` (``-f csv``).
--bench FILE  a file holding bench.py's JSON line: the roofline kernel's
              dispatches are picked out of the trace by name, workgroup size and
              total grid size, and their average duration is set beside the
              latency bench.py measured with HIP events.
--replay FILE the JSON line of ``tuner --replay`` (the same kernel run alone,
              then the copy kernel over a known number of bytes).
--fetch/--write DIR  ``-f csv`` output of a ``--pmc FETCH_SIZE`` and a
              ``--pmc WRITE_SIZE`` run of that replay. The counters read KiB per
              dispatch; each is scaled by known bytes / counted bytes of the copy
              kernel in the same run.

--sq DIR --replay FILE  SQ-counter mode: ``-f csv`` output of a ``--pmc``
              pass of SQ counters over that replay (``--sq`` once per pass);
              writes per-dispatch, per-wave and per-MFMA figures instead.

The output ends with a JSON block (``traffic``) that bench.py reads back: it
names the kernel, its launch shape and a hash of the kernel's source files and
of the schedule rules, so a later change to the kernel or its geometry voids
the figure.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sqlite3
import statistics
import sys
from collections import defaultdict

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")

# kernel name prefix -> the source files that define it
PEAK_FP32_TFLOPS = 157.3  # MI355X dense fp32 (vector and MFMA), 256 CUs at 2.4 GHz
PEAK_BF16_TFLOPS = 2516.6  # MI355X dense bf16 MFMA
PEAK_HBM_TBPS = 8.0        # MI355X HBM3E

_KERNEL_SOURCES = {
    "direct_f32_kernel": ["k_direct*"],
    "depthwise_f32_kernel": ["k_depthwise*"],
    "depthwise_q4_kernel": ["k_depthwise*"],
    "igemm_bf16_kernel": ["k_igemm_bf16*"],
    "igemm_f32_kernel": ["k_igemm_f32*"],
}


def kernel_source_hash(kernel: str) -> str | None:
    """sha256 over the sources of the family that `kernel` belongs to, plus the
    shared headers and the schedule rules that set every launch's geometry
    (tile sizes, LDS pitches); None for a kernel this library does not define."""
    base = kernel.replace("void ", "").split("<")[0].split("(")[0].split("::")[-1]
    pats = _KERNEL_SOURCES.get(base)
    if not pats:
        return None
    files = sorted(set(f for p in pats + ["k_util.h", "ct_internal.h", "schedule.cpp"] for f in glob.glob(os.path.join(CSRC, p))))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _lds_ok(traced, requested) -> bool:
    """A rocpd trace lists a dispatch's LDS as allocated, rounded up to the
    allocation granule (accept up to 1 KiB above the bytes the launch asked
    for); a csv trace reports 0 for LDS sized at launch (not a mismatch)."""
    if requested is None or not traced:
        return True
    return requested <= traced <= requested + 1024


def short_name(name: str) -> str:
    return name.replace("void ", "").split("(")[0]


# ---------------------------------------------------------------- trace input
class Trace:
    """Kernel dispatches of one profiler run: (name, grid items, wg size, duration ns)."""

    def __init__(self, directory: str):
        dbs = sorted(glob.glob(os.path.join(directory, "**", "*.db"), recursive=True))
        self.db = sqlite3.connect(dbs[0]) if dbs else None
        self.rows = None
        if self.db is None:
            self.rows = []
            for path in sorted(glob.glob(os.path.join(directory, "**", "*kernel_trace.csv"), recursive=True)):
                with open(path) as fh:
                    for r in csv.DictReader(fh):
                        grid = _int(r, "Grid_Size") or (_int(r, "Grid_Size_X") * max(_int(r, "Grid_Size_Y"), 1)
                                                        * max(_int(r, "Grid_Size_Z"), 1))
                        wg = _int(r, "Workgroup_Size") or (_int(r, "Workgroup_Size_X")
                                                           * max(_int(r, "Workgroup_Size_Y"), 1)
                                                           * max(_int(r, "Workgroup_Size_Z"), 1))
                        self.rows.append((r.get("Kernel_Name", ""), grid, wg, _int(r, "LDS_Block_Size", "Lds_Size"),
                                          _int(r, "End_Timestamp") - _int(r, "Start_Timestamp")))

    def by_stream(self, kernel: str, wg: int | None, grid: int | None, lds: int | None = None):
        """{stream id: [durations]} of the matching dispatches (rocpd traces only)."""
        out = defaultdict(list)
        if self.db is None:
            return out
        q = ("SELECT name, workgroup_x * workgroup_y * workgroup_z, grid_x * grid_y * grid_z, lds_size, "
             "stream_id, duration FROM kernels WHERE name LIKE ?")
        for n, w, g, l, st, d in self.db.execute(q, ("%" + kernel + "%",)):
            if (kernel in n.replace("void ", "") and (wg is None or w == wg) and (grid is None or g == grid)
                    and _lds_ok(l, lds)):
                out[st].append(d)
        return out

    def per_kernel(self):
        """[(short name, dispatches, total ns, mean ns)] sorted by total time."""
        by = defaultdict(lambda: [0, 0])
        if self.db is not None:
            q = "SELECT name, count(*), sum(duration) FROM kernels GROUP BY name"
            for name, n, tot in self.db.execute(q):
                e = by[short_name(name)]
                e[0] += n
                e[1] += tot
        else:
            for name, _, _, _, d in self.rows:
                e = by[short_name(name)]
                e[0] += 1
                e[1] += d
        out = [(k, n, tot, tot / n) for k, (n, tot) in by.items()]
        return sorted(out, key=lambda r: -r[2])

    def durations(self, kernel: str, wg: int | None, grid: int | None, lds: int | None = None):
        """Durations (ns) of the dispatches of `kernel` with that shape (and LDS bytes)."""
        if self.db is not None:
            q = ("SELECT name, workgroup_x * workgroup_y * workgroup_z, grid_x * grid_y * grid_z, lds_size, "
                 "duration FROM kernels WHERE name LIKE ?")
            rows = self.db.execute(q, ("%" + kernel + "%",)).fetchall()
        else:
            rows = [(n, w, g, l, d) for n, g, w, l, d in self.rows if kernel in n]
        return [d for n, w, g, l, d in rows
                if kernel in n.replace("void ", "") and (wg is None or w == wg) and (grid is None or g == grid)
                and _lds_ok(l, lds)]


def _int(r, *names):
    for n in names:
        if n in r and r[n] not in (None, ""):
            return int(float(r[n]))
    return 0


def counter_per_dispatch(directory: str, counter: str):
    """{short kernel name: [value per dispatch]} from a --pmc CSV run."""
    out = defaultdict(list)
    for path in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)):
        with open(path) as fh:
            per = defaultdict(float)
            names = {}
            for r in csv.DictReader(fh):
                if r.get("Counter_Name") != counter:
                    continue
                key = r.get("Dispatch_Id") or r.get("Correlation_Id")
                per[key] += float(r["Counter_Value"])
                names[key] = r.get("Kernel_Name", "")
            for key, v in per.items():
                out[short_name(names[key])].append(v)
    return out


# ---------------------------------------------------------------- summary
def _read_json_line(path: str, key: str):
    if not path:
        return None
    with open(path) as fh:
        for line in fh:
            line = line.strip()
            if line.startswith("{") and key in line:
                return json.loads(line)
    return None


def summarize(trace_dir, bench=None, replay=None, fetch_dir=None, write_dir=None, cmds=(), traced_bench=None) -> str:
    """Kernel table of a trace; with `bench` (bench.py's JSON line) the trace
    durations of the kernel and launch shape it names, set beside its HIP-event
    latency. `traced_bench` is the line the traced run itself printed, when
    `bench` comes from an untraced run of the same command: the tracer adds
    time to every launch, which reorders near-equal candidates, so the two
    runs can name different winners; every candidate is screened on every
    share in both, so the untraced winner's launches are in the trace."""
    tr = Trace(trace_dir)
    lines = ["# rocprofv3 kernel summary", ""]
    if tr.db is None and not tr.rows:
        lines += ["No trace (no rocpd database or kernel_trace.csv) under %s." % trace_dir, ""]
    if cmds:
        lines += ["Commands (run from the repository root):", "", "```"] + list(cmds) + ["```", ""]
    rows = tr.per_kernel()
    total = sum(r[2] for r in rows)
    lines += ["Trace: %d dispatches, total kernel time %.3f ms." % (sum(r[1] for r in rows), total / 1e6), "",
              "| kernel | dispatches | total ms | share | avg us |", "|---|---|---|---|---|"]
    for name, n, tot, mean in rows[:25]:
        lines.append("| `%s` | %d | %.3f | %.1f%% | %.2f |" % (name, n, tot / 1e6, 100.0 * tot / max(total, 1),
                                                                mean / 1e3))
    block = {}
    if bench and "roofline" in bench:
        rf = bench["roofline"]
        shape = rf.get("launch_shape", {})
        kname = rf.get("kernel", "")
        threads, blocks = shape.get("threads"), shape.get("blocks")
        grid = blocks * threads if blocks and threads else None
        durs = tr.durations(kname, threads, grid, shape.get("lds_bytes"))
        lines += ["", "## Roofline kernel", "",
                  "bench.py%s names `%s` (layer %s, %s blocks x %s threads, LDS %s bytes, knobs %s), "
                  "%.3f GFLOP per launch."
                  % (" (untraced run)" if traced_bench else "", kname, rf.get("layer"), blocks, threads,
                     shape.get("lds_bytes"), ",".join(str(v) for v in shape.get("knobs", {}).values()),
                     rf.get("flops_per_launch", 0) / 1e9), ""]
        if traced_bench and "roofline" in traced_bench:
            tr_rf = traced_bench["roofline"]
            tr_sh = tr_rf.get("launch_shape", {})
            same = tr_rf.get("kernel") == kname and tr_sh.get("knobs") == shape.get("knobs")
            lines += ["The traced run of the same command named %s (%.3f us by its HIP events, which hold "
                      "the tracer's per-launch cost); the rows below are the untraced winner's launches in "
                      "the trace." % ("the same schedule" if same else "`%s` knobs %s" % (
                          tr_rf.get("kernel"), ",".join(str(v) for v in tr_sh.get("knobs", {}).values())),
                          tr_rf.get("latency_us", 0.0)), ""]
        if durs:
            avg = statistics.mean(durs) / 1e3
            groups = tr.by_stream(kname, threads, grid, shape.get("lds_bytes"))
            if len(groups) > 1:
                # the same candidate list is timed on every CU share: one stream per share
                lines += ["The kernel ran on %d streams (one per CU share and client); per stream:" % len(groups),
                          "", "| stream | launches | avg us |", "|---|---|---|"]
                for st, v in sorted(groups.items(), key=lambda kv: statistics.mean(kv[1])):
                    lines.append("| %s | %d | %.3f |" % (st, len(v), statistics.mean(v) / 1e3))
                durs = min(groups.values(), key=statistics.mean)
                lines += ["", "The fastest streams are the full-GPU ones (the roofline's share); the rows below "
                              "use the fastest.", ""]
                avg = statistics.mean(durs) / 1e3
            if shape.get("kernels", 1) > 1:
                red = tr.durations("split_reduce_kernel", None, None)
                lines += ["The schedule splits the reduction, so bench.py's latency covers this kernel plus "
                          "`split_reduce_kernel`; the trace holds %d launches of the latter from all split "
                          "schedules (avg %.3f us)." % (len(red), statistics.mean(red) / 1e3 if red else 0.0), ""]
            lines += ["| source | launches | avg us | median us |", "|---|---|---|---|",
                      "| rocprofv3 kernel trace | %d | %.3f | %.3f |" % (len(durs), avg,
                                                                      statistics.median(durs) / 1e3),
                      "| bench.py HIP events (median of repeat means) | - | %.3f | - |" % rf.get("latency_us", 0.0),
                      "", "From the trace average: %.2f TFLOP/s, %.1f%% of %.1f %s." % (
                          rf["flops_per_launch"] / (avg * 1e-6) / 1e12,
                          100.0 * rf["flops_per_launch"] / (avg * 1e-6) / 1e12 / rf["peak"], rf["peak"],
                          rf.get("unit", ""))]
            if rf.get("latency_us", 0.0) > avg:
                lines.append("(The bench's first launch of each repeat follows a host-side event record, so "
                             "its HIP-event mean also holds launch gaps that the trace does not.)")
        else:
            lines.append("No dispatch of that kernel with that shape is in the trace.")
    if replay:
        lines += ["", "## Replay (kernel alone)", "",
                  "`%s`, %d launches at %g%% of the CUs: %.3f us by HIP events, %.2f TFLOP/s." % (
                      replay["kernel"], replay["launches"], 100 * replay["fraction"], replay["latency_us"],
                      replay["tflops"])]
        sh = replay["schedule"]
        rdurs = tr.durations(replay["kernel"], sh.get("threads"), sh.get("blocks", 0) * sh.get("threads", 0),
                             sh.get("lds_bytes"))
        if rdurs:
            tavg = statistics.mean(rdurs) / 1e3
            ttf = replay["tflops"] * replay["latency_us"] / tavg  # the launch's FLOP over the trace average
            lines.append("Trace of the replay: %d launches, avg %.3f us, median %.3f us; from the average %.2f "
                         "TFLOP/s = %.1f%% of the fp32 peak scaled to the share (%.1f x %g)." % (
                             len(rdurs), tavg, statistics.median(rdurs) / 1e3, ttf,
                             100 * ttf / (PEAK_FP32_TFLOPS * replay["fraction"]), PEAK_FP32_TFLOPS,
                             replay["fraction"]))
            if replay.get("bytes_moved"):
                # |x| + |w| + |y| once per launch: the bound of the memory-bound families
                tbps = replay["bytes_moved"] / (tavg * 1e-6) / 1e12
                lines.append("Algorithmic bytes (|x| + |w| + |y|) %d per launch: from the trace average %.2f TB/s "
                             "= %.1f%% of the %.1f TB/s HBM peak (which does not scale with the CU share)." % (
                                 replay["bytes_moved"], tbps, 100 * tbps / PEAK_HBM_TBPS, PEAK_HBM_TBPS))
                if replay.get("dtype") == "bf16":
                    lines.append("The bf16 MFMA side: %.2f TFLOP/s = %.2f%% of %.1f TFLOP/s x %g." % (
                        ttf, 100 * ttf / (PEAK_BF16_TFLOPS * replay["fraction"]), PEAK_BF16_TFLOPS,
                        replay["fraction"]))
            if sh.get("kernels", 1) > 1:
                red = tr.durations("split_reduce_kernel", None, None)
                if red:
                    both = statistics.mean(rdurs) + statistics.mean(red)
                    lines.append("The schedule splits the reduction: each run is the kernel above plus "
                                 "`split_reduce_kernel` (avg %.3f us over %d launches), %.3f us together "
                                 "(%.2f TFLOP/s)." % (statistics.mean(red) / 1e3, len(red), both / 1e3,
                                                      replay["tflops"] * replay["latency_us"] / (both / 1e3)))
    if replay and fetch_dir and write_dir:
        t = traffic_block(replay, fetch_dir, write_dir)
        if t is not None:
            lines += ["", "## HBM traffic (counters)", "",
                      "| counter | copy kernel KiB (known %d MiB) | scale | kernel KiB per launch (median of %d) "
                      "| kernel bytes per launch |" % (replay["copy_bytes_each_way"] >> 20, t["n"]),
                      "|---|---|---|---|---|",
                      "| FETCH_SIZE | %.0f | %.4f | %.1f | %.0f |" % (t["copy_fetch_kib"], t["scale_f"], t["fetch_kib"],
                                                                 t["block"]["fetch_bytes"]),
                      "| WRITE_SIZE | %.0f | %.4f | %.1f | %.0f |" % (t["copy_write_kib"], t["scale_w"], t["write_kib"],
                                                                 t["block"]["write_bytes"])]
            block = t["block"]
        else:
            lines += ["", "Counter runs incomplete: traffic not derived."]
    if block:
        lines += ["", "```json", json.dumps({"traffic": block}), "```"]
    return "\n".join(lines) + "\n"


def _json_blocks(text: str):
    """Every fenced json block of a summary, parsed (unparsable ones skipped)."""
    pos = 0
    while True:
        start = text.find("```json\n", pos)
        if start < 0:
            return
        end = text.find("```", start + 8)
        if end < 0:
            return
        try:
            yield json.loads(text[start + 8:end])
        except ValueError:
            pass
        pos = end + 3


def find_traffic(profiles_dir: str, kernel: str, shape: dict):
    """Traffic bytes per launch for `kernel` with this launch shape from a
    summary under profiles_dir, or None (no summary, another shape, or the
    kernel's sources changed since the counters were taken)."""
    want = kernel_source_hash(kernel)
    if want is None:
        return None
    for path in sorted(glob.glob(os.path.join(profiles_dir, "*.md"))):
        with open(path) as fh:
            text = fh.read()
        for doc in _json_blocks(text):
            blk = doc.get("traffic") if isinstance(doc, dict) else None
            if not isinstance(blk, dict):
                continue
            if (blk.get("kernel") == kernel and blk.get("threads") == shape.get("threads")
                    and blk.get("blocks") == shape.get("blocks") and blk.get("knobs") == shape.get("knobs")
                    and blk.get("source_hash") == want):
                return blk
    return None


def traffic_block(replay: dict, fetch_dir: str, write_dir: str):
    """(FETCH, WRITE) medians in KiB, copy-kernel scales and the traffic block
    of one replayed schedule, or None if a counter run is incomplete."""
    k = short_name(replay["kernel"])
    f = counter_per_dispatch(fetch_dir, "FETCH_SIZE")
    w = counter_per_dispatch(write_dir, "WRITE_SIZE")
    kf = [v for name, vs in f.items() if k in name for v in vs]
    kw = [v for name, vs in w.items() if k in name for v in vs]
    cf = [v for name, vs in f.items() if "copy_kernel" in name for v in vs]
    cw = [v for name, vs in w.items() if "copy_kernel" in name for v in vs]
    nbytes = replay.get("copy_bytes_each_way", 0)
    if not (kf and kw and cf and cw and nbytes):
        return None
    sf = nbytes / (max(cf) * 1024.0)
    sw = nbytes / (max(cw) * 1024.0)
    fetch = statistics.median(kf) * 1024.0 * sf
    write = statistics.median(kw) * 1024.0 * sw
    sched = replay["schedule"]
    block = {"kernel": replay["kernel"], "layer": replay["layer"], "threads": sched.get("threads"),
             "blocks": sched.get("blocks"), "lds_bytes": sched.get("lds_bytes"),
             "knobs": sched.get("knobs"), "fetch_bytes": fetch, "write_bytes": write,
             "traffic_bytes": fetch + write, "source_hash": kernel_source_hash(replay["kernel"])}
    return {"fetch_kib": statistics.median(kf), "write_kib": statistics.median(kw), "n": len(kf),
            "copy_fetch_kib": max(cf), "copy_write_kib": max(cw), "scale_f": sf, "scale_w": sw, "block": block}


def traffic_table(entries, cmds=()) -> str:
    """Summary of several replayed schedules' counter runs: one row and one
    traffic block each. entries: (replay dict, fetch dir, write dir)."""
    lines = ["# HBM traffic of candidate schedules (FETCH_SIZE / WRITE_SIZE counters)", "",
             "Each schedule was replayed alone (back-to-back launches on slot 0 of its share) under one "
             "counter per run; the copy kernel of the same run, over a buffer of known size, calibrates "
             "the counters. (Kernel times under counter collection are not representative and are not "
             "listed.)", "", "Commands (one pair per schedule, `$ARG` = layer:family:knobs as listed):", ""]
    lines += ["    " + c for c in cmds]
    lines += ["", "| layer | kernel | knobs | launches | FETCH KiB | WRITE KiB | scale F / W | traffic bytes |",
              "|---|---|---|---|---|---|---|---|"]
    blocks = []
    for rep, fdir, wdir in entries:
        t = traffic_block(rep, fdir, wdir)
        knobs = ",".join(str(v) for v in rep["schedule"]["knobs"].values())
        if t is None:
            lines.append("| %s | `%s` | %s | - | incomplete | | | |" % (rep["layer"], rep["kernel"], knobs))
            continue
        lines.append("| %s | `%s` | %s | %d | %.1f | %.1f | %.4f / %.4f | %.0f |" % (
            rep["layer"], rep["kernel"], knobs, t["n"], t["fetch_kib"], t["write_kib"], t["scale_f"], t["scale_w"],
            t["block"]["traffic_bytes"]))
        blocks.append(t["block"])
    for b in blocks:
        lines += ["", "```json", json.dumps({"traffic": b}), "```"]
    return "\n".join(lines) + "\n"


SQ_COUNTERS = ("SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_LDS",
               "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_F32")
# Units of the SQ counters these summaries use, from rocprofiler's counter
# definitions: the per-wave time counters count quad-cycles (4 clocks; a
# wave issues at most one instruction per quad-cycle, so the ACTIVE counters
# track the INSTS counters), the MFMA-busy and bank-conflict counters clocks.
# The summary converts all of them to clocks.
SQ_UNITS = {"SQ_WAVES": ("waves", 1), "SQ_WAVE_CYCLES": ("quad-cycles", 4), "SQ_INSTS_LDS": ("instructions", 1),
            "SQ_LDS_BANK_CONFLICT": ("cycles", 1), "SQ_WAIT_INST_LDS": ("quad-cycles", 4),
            "SQ_VALU_MFMA_BUSY_CYCLES": ("cycles", 1), "SQ_INSTS_VALU_MFMA_F32": ("instructions", 1),
            "SQ_WAIT_ANY": ("quad-cycles", 4), "SQ_WAIT_INST_ANY": ("quad-cycles", 4),
            "SQ_ACTIVE_INST_ANY": ("quad-cycles", 4), "SQ_ACTIVE_INST_VALU": ("quad-cycles", 4),
            "SQ_ACTIVE_INST_LDS": ("quad-cycles", 4), "SQ_ACTIVE_INST_VMEM": ("quad-cycles", 4),
            "SQ_ACTIVE_INST_SCA": ("quad-cycles", 4), "SQ_ACTIVE_INST_MISC": ("quad-cycles", 4),
            "SQ_INSTS_VALU": ("instructions", 1), "SQ_INSTS_SALU": ("instructions", 1),
            "SQ_INSTS_VMEM": ("instructions", 1)}
SQ_CLOCK_GHZ = 2.4  # MI355X peak engine clock


def _sq_medians(sq_dirs, short):
    """{counter: median per dispatch} over every SQ counter found in the
    --pmc runs (one directory per pass), and the dispatch count."""
    med, n_disp = {}, 0
    for d in sq_dirs:
        names = set()
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as fh:
                names |= {r.get("Counter_Name", "") for r in csv.DictReader(fh)}
        for c in sorted(n for n in names if n.startswith("SQ_")):
            vals = next((v for k, v in counter_per_dispatch(d, c).items() if short in k), [])
            if vals:
                med.setdefault(c, statistics.median(vals))
                n_disp = max(n_disp, len(vals))
    return med, n_disp


def sq_summary(replay: dict, sq_dirs, cmds=()) -> str:
    """SQ counters of one replayed fp32 MFMA schedule (one --pmc pass per
    directory): median per dispatch, per wave and per MFMA instruction,
    against the MFMAs the layer's FLOPs need (2048 FLOP per 16x16x4, 4096 per
    32x32x2), and where the waves' time goes."""
    if isinstance(sq_dirs, str):
        sq_dirs = [sq_dirs]
    short = replay["kernel"]
    med, n_disp = _sq_medians(sq_dirs, short)
    order = [c for c in SQ_COUNTERS if c in med] + sorted(c for c in med if c not in SQ_COUNTERS and c in SQ_UNITS)
    unknown = sorted(c for c in med if c not in SQ_UNITS)
    knobs = ",".join(str(v) for v in replay["schedule"]["knobs"].values())
    mfma_flops = 2048 if replay["schedule"]["knobs"].get("mfma", 16) == 16 else 4096
    need = replay["flops"] / mfma_flops
    lines = ["# SQ counters of `%s` on %s (knobs %s) at %g %% of the CUs" % (short, replay["layer"], knobs,
                                                                          100 * replay["fraction"]),
             "", "Replayed alone; medians over %d dispatches, summed over the device. Command%s (run from the "
             "repository root, %d SQ counters in %d pass%s):" % (
                 n_disp, "s" if len(cmds) > 1 else "", len(med), len(sq_dirs), "es" if len(sq_dirs) > 1 else ""),
             "", "```"]
    lines += list(cmds) + ["```", ""]
    if unknown:
        lines += ["Collected but not reported (no unit defined here): %s." % ", ".join(unknown), ""]
    lines += ["| counter | unit | per dispatch | per wave | per MFMA | clocks per wave |",
                           "|---|---|---|---|---|---|"]
    waves = med.get("SQ_WAVES") or 0
    mf = med.get("SQ_INSTS_VALU_MFMA_F32") or 0
    for c in order:
        v = med[c]
        unit, clocks = SQ_UNITS[c]
        lines.append("| %s | %s | %.0f | %s | %s | %s |" % (
            c, unit, v, "%.1f" % (v / waves) if waves else "-",
            "%.2f" % (v / mf) if mf and c != "SQ_WAVES" else "-",
            "%.0f" % (clocks * v / waves) if waves and unit.endswith("cycles") else "-"))
    life = 4 * med.get("SQ_WAVE_CYCLES", 0) / waves if waves else 0
    if mf and waves:
        lines += ["", "The layer needs %.0f MFMAs of %d FLOP; the kernel issues %.0f (%+.1f %%: tile padding)." % (
            need, mfma_flops, mf, 100 * (mf / need - 1))]
        if life and "SQ_VALU_MFMA_BUSY_CYCLES" in med:
            busy = med["SQ_VALU_MFMA_BUSY_CYCLES"]
            bc = med.get("SQ_LDS_BANK_CONFLICT", 0)
            # (the replay's own HIP-event latency is no check here: counter
            # collection serialises the dispatches and inflates it)
            lines.append("A wave lives %.0f clocks (%.2f us at %.1f GHz); its MFMAs keep the MFMA pipe busy for "
                         "%.0f of them (%.1f %%), bank conflicts stall LDS for %.0f (%.1f %%)." % (
                             life, life / (1e3 * SQ_CLOCK_GHZ), SQ_CLOCK_GHZ,
                             busy / waves, 100 * busy / waves / life, bc / waves, 100 * bc / waves / life))
        lds = med.get("SQ_INSTS_LDS", 0)
        if lds:
            lines.append("LDS bank-conflict cycles per LDS instruction: %.2f (%.0f instructions per wave)." % (
                med.get("SQ_LDS_BANK_CONFLICT", 0) / lds, lds / waves))
    if life and all(c in med for c in ("SQ_ACTIVE_INST_ANY", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY")):
        part = [100 * 4 * med[c] / waves / life for c in ("SQ_ACTIVE_INST_ANY", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY")]
        lines.append("Of a wave's life, %.0f %% goes to issuing instructions (SQ_ACTIVE_INST_ANY), %.0f %% to "
                     "waiting for a dependency: memory, LDS, a barrier (SQ_WAIT_ANY), and %.0f %% to waiting "
                     "for its turn to issue (SQ_WAIT_INST_ANY)." % tuple(part))
    return "\n".join(lines) + "\n"


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", default=None)
    ap.add_argument("--bench", default=None, help="file holding bench.py's JSON line")
    ap.add_argument("--traced-bench", default=None,
                    help="file holding the JSON line of the traced run, when --bench is an untraced run")
    ap.add_argument("--replay", default=None, help="file holding tuner --replay's JSON line")
    ap.add_argument("--fetch", default=None)
    ap.add_argument("--write", default=None)
    ap.add_argument("--entry", action="append", default=[], metavar="REPLAY_JSON:FETCH_DIR:WRITE_DIR",
                    help="traffic-table mode: one replayed schedule and its two counter runs")
    ap.add_argument("--sq", action="append", default=[],
                    help="SQ-counter mode: a --pmc directory of one replay (with --replay); repeat for more passes")
    ap.add_argument("--out", default=None)
    ap.add_argument("--cmd", action="append", default=[])
    a = ap.parse_args(argv)
    if a.sq:
        rep = _read_json_line(a.replay, '"kernel"')
        if rep is None:
            ap.error("--sq needs --replay")
        text = sq_summary(rep, a.sq, a.cmd)
    elif a.entry:
        entries = []
        for e in a.entry:
            rj, fd, wd = e.split(":")
            rep = _read_json_line(rj, '"kernel"')
            if rep is not None:
                entries.append((rep, fd, wd))
        text = traffic_table(entries, a.cmd)
    else:
        if not a.trace:
            ap.error("--trace is required without --entry")
        text = summarize(a.trace, _read_json_line(a.bench, '"metric"'), _read_json_line(a.replay, '"kernel"'),
                         a.fetch, a.write, a.cmd, _read_json_line(a.traced_bench, '"metric"'))
    if a.out:
        with open(a.out, "w") as fh:
            fh.write(text)
    sys.stdout.write(text)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
