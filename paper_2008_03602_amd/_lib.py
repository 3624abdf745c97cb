"""ctypes binding of libconvtune.so: argument marshalling only.

Every function here has the name of the C entry point it calls (see
``include/convtune.h``), turns Python/numpy/torch arguments into the C
structs and pointers, raises ``CtError`` on a negative return code, and
returns the outputs as numpy arrays. No step of the tuning path runs here.
Loading fails loudly when the library is missing: there is no fallback.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import threading
from typing import Iterable, List, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libconvtune.so")

CT_OK, CT_E_ARG, CT_E_HIP, CT_E_NOINIT, CT_E_OOM, CT_E_NODEV = 0, -1, -2, -3, -4, -5
CT_E_TIMEOUT, CT_E_CLIENT, CT_E_STOPPED = -6, -7, -8
S_OK, S_INVALID, S_LAUNCH, S_TIMEOUT, S_WRONG_ANSWER = 0, 1, 2, 3, 4
STATUS_NAMES = {0: "ok", 1: "invalid", 2: "launch_error", 3: "timeout", 4: "wrong_answer"}
MASK_WORDS = 8
MAX_KNOBS = 15

c_i32, c_i64, c_u32, c_u64, c_f32, c_f64 = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                            ctypes.c_uint64, ctypes.c_float, ctypes.c_double)
P = ctypes.POINTER


class CtError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("libconvtune error %d: %s" % (code, msg))
        self.code = code


class ct_op(ctypes.Structure):
    _fields_ = [(n, c_i32) for n in ("n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h",
                                     "pad_w", "dil_h", "dil_w", "groups", "dtype", "layout")]


class ct_schedule(ctypes.Structure):
    _fields_ = [("family", c_i32), ("knob", c_i32 * MAX_KNOBS)]


class ct_measure_opts(ctypes.Structure):
    _fields_ = [("warmup", c_i32), ("repeats", c_i32), ("launches", c_i32), ("batch", c_i32),
                ("timeout_ms", c_f32), ("interleave", c_i32)]


class ct_verify(ctypes.Structure):
    _fields_ = [("y_ref", ctypes.c_void_p), ("tol", c_f32)]


class ct_tune_job(ctypes.Structure):
    _fields_ = [("op", ct_op), ("x", ctypes.c_void_p), ("w", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("cands", P(ct_schedule)), ("n_cands", c_i32), ("verify", ct_verify),
                ("lat1_us", P(c_f32)), ("status1", P(c_i32)), ("top_t", c_i32),
                ("top_pos", P(c_i32)), ("lat2_us", P(c_f32)), ("n_top", c_i32), ("winner_pos", c_i32),
                ("winner_lat_us", c_f32), ("t_start_s", c_f64), ("t_end_s", c_f64), ("layer_id", c_i32),
                ("skip", P(ctypes.c_uint8)), ("rc", c_i32)]


class ct_client(ctypes.Structure):
    _fields_ = [("cu_mask", c_u32 * MASK_WORDS), ("host_core", c_i32), ("jobs", P(ct_tune_job)),
                ("n_jobs", c_i32), ("rc", c_i32), ("t_start_s", c_f64), ("t_end_s", c_f64),
                ("n_measured", c_i64), ("log_path", ctypes.c_char_p), ("cands_per_s", c_f64)]


class ct_test_hooks(ctypes.Structure):
    _fields_ = [("delay_us", c_i32), ("throw_client", c_i32), ("throw_after_jobs", c_i32),
                ("stop_after_records", c_i64)]


class ct_search_opts(ctypes.Structure):
    _fields_ = [("seed", c_u64), ("batch", c_i32), ("budget", c_i32), ("patience", c_i32), ("sa_chains", c_i32),
                ("sa_steps", c_i32), ("explore", c_f32), ("eps", c_f32), ("sa_temp", c_f32), ("cus", c_i32)]


class ct_search_result(ctypes.Structure):
    _fields_ = [("n_measured", c_i32), ("rounds", c_i32), ("stopped_early", c_i32), ("winner", c_i32),
                ("winner_lat_us", c_f32), ("pad_", c_f32), ("propose_s", c_f64), ("measure_s", c_f64)]


_SIGS = {
    "ct_init": (c_i32, [c_i32]),
    "ct_num_cus": (c_i32, []),
    "ct_shutdown": (None, []),
    "ct_last_error": (ctypes.c_char_p, []),
    "ct_build_cu_mask": (c_i32, [c_i32, c_f64, c_i32, P(c_u32), c_i32]),
    "ct_cu_mask": (c_i32, [c_f64, c_i32, P(c_u32), c_i32]),
    "ct_grid_info": (c_i32, [c_i32, P(c_i32), P(c_i64)]),
    "ct_grid_size": (c_i32, [P(ct_op), c_i32, P(c_i64)]),
    "ct_set_reference": (c_i32, [P(ct_op), P(c_f64)]),
    "ct_throughput": (c_i32, [P(ct_client), c_i32, P(c_f64)]),
    "ct_tune_split": (c_i32, [P(ct_tune_job), P(c_u32), c_i32, c_i32, P(ctypes.c_void_p), P(ct_measure_opts),
                              P(ct_measure_opts), c_f32, P(c_f64)]),
    "ct_stream_count": (c_i32, []),
    "ct_test_xcd_band": (c_i32, [c_i32, P(c_i32)]),
    "ct_test_run_clients": (c_i32, [P(ct_client), c_i32, P(ct_tune_job), c_i32, P(ct_test_hooks), P(c_i32)]),
    "ct_test_watchdog": (c_i32, [c_i32, P(c_i32), P(c_f64), c_f64, c_f64, c_f64, P(c_i32), P(c_i32)]),
    "ct_knob_values": (c_i32, [c_i32, c_i32, P(c_i32), c_i32, P(c_i32)]),
    "ct_grid_decode": (c_i32, [c_i32, c_i64, P(ct_schedule)]),
    "ct_grid_encode": (c_i32, [P(ct_schedule), P(c_i64)]),
    "ct_validate": (c_i32, [P(ct_op), P(ct_schedule)]),
    "ct_launch_shape": (c_i32, [P(ct_op), P(ct_schedule), P(c_i32), P(c_i32), P(c_i64), P(c_i32)]),
    "ct_kernel_name": (c_i32, [P(ct_op), P(ct_schedule), ctypes.c_char_p, c_i32]),
    "ct_valid_space": (c_i32, [P(ct_op), P(ct_schedule), c_i64, P(c_i64)]),
    "ct_sample": (c_i32, [P(ct_op), c_u64, c_i32, c_i32, c_i32, P(ct_schedule), P(c_i32)]),
    "ct_sample_uniform": (c_i32, [P(ct_op), c_u64, c_i32, c_i32, c_i32, P(ct_schedule), P(c_i32)]),
    "conv2d_run": (c_i32, [P(ct_op), P(ct_schedule), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                           P(c_u32), c_i32]),
    "conv2d_run_noalloc": (c_i32, [P(ct_op), P(ct_schedule), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p]),
    "measure_candidates": (c_i32, [P(ct_op), P(ct_schedule), c_i32, c_f64, P(ct_measure_opts),
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, P(c_f32), P(c_i32)]),
    "measure_candidates_mask": (c_i32, [P(ct_op), P(ct_schedule), c_i32, P(c_u32), c_i32,
                                        P(ct_measure_opts), P(ct_verify), ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, P(c_f32), P(c_i32), P(c_f32)]),
    "ct_top_t": (c_i32, [P(c_f32), P(c_i32), c_i32, c_i32, P(c_i32), P(c_i32)]),
    "ct_select_winner": (c_i32, [P(c_f32), P(c_i32), c_i32, c_f32, P(c_i32)]),
    "ct_tune_clients": (c_i32, [P(ct_client), c_i32, P(ct_measure_opts), P(ct_measure_opts), c_f32]),
    "ct_tune_shared": (c_i32, [P(ct_client), c_i32, P(ct_tune_job), c_i32, P(ct_measure_opts),
                               P(ct_measure_opts), c_f32, P(c_i32)]),
    "ct_cross_eval": (c_i32, [P(ct_op), P(ct_schedule), c_i32, P(c_u32), c_i32, c_i32, P(ct_measure_opts),
                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, P(c_f32)]),
    "ct_search_propose": (c_i32, [P(ct_op), P(ct_schedule), P(c_f32), P(c_i32), c_i32, P(ct_search_opts), c_i32,
                                  P(ct_schedule), c_i32, P(c_i32)]),
    "ct_search": (c_i32, [P(ct_op), P(ct_search_opts), P(c_u32), c_i32, P(ct_measure_opts), P(ct_measure_opts),
                          c_i32, c_f32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, P(ct_schedule), P(c_f32),
                          P(c_i32), P(ct_search_result)]),
    "ct_probe_cus": (c_i32, [P(c_u32), c_i32, c_i32, P(c_i32), c_i32, P(c_i32)]),
    "ct_probe_empty": (c_i32, [P(c_u32), c_i32, c_i32, P(ct_measure_opts), P(c_f32)]),
    "ct_probe_copy": (c_i32, [P(c_u32), c_i32, ctypes.c_void_p, ctypes.c_void_p, c_i64, P(ct_measure_opts),
                              P(c_f32)]),
}

_lock = threading.Lock()
_lib = None


def lib():
    """The loaded library (built in-tree by ``paper_2008_03602_amd.build``)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError("libconvtune.so is not built (%s); run `python -m "
                                   "paper_2008_03602_amd.build` first" % LIB_PATH)
            h = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in _SIGS.items():
                f = getattr(h, name)
                f.restype = res
                f.argtypes = args
            _lib = h
            # streams, events and workspaces go back before the HIP runtime's
            # own teardown at process exit (ct_shutdown is safe to call twice)
            atexit.register(h.ct_shutdown)
    return _lib


def _check(rc: int) -> int:
    if rc < 0:
        raise CtError(rc, lib().ct_last_error().decode(errors="replace"))
    return rc


def _arr(a, ctype):
    return a.ctypes.data_as(P(ctype))


def _ptr(t) -> int:
    """Device address of a torch tensor (or an int address)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


# ---------------------------------------------------------------- structs
def make_op(op) -> ct_op:
    """ct_op from a workloads.Op (or any object with the same fields, or a 16-tuple)."""
    vals = op.as_tuple() if hasattr(op, "as_tuple") else tuple(op)
    return ct_op(*vals)


def make_schedule(family: int, knobs: Sequence[int]) -> ct_schedule:
    s = ct_schedule()
    s.family = family
    for i, v in enumerate(knobs):
        s.knob[i] = int(v)
    return s


def schedule_tuple(s: ct_schedule):
    return (int(s.family),) + tuple(int(v) for v in s.knob)


def schedule_array(scheds: Sequence) -> ctypes.Array:
    arr = (ct_schedule * max(len(scheds), 1))()
    for i, s in enumerate(scheds):
        arr[i] = s if isinstance(s, ct_schedule) else make_schedule(s[0], s[1:])
    return arr


def make_opts(warmup=2, repeats=5, launches=10, batch=16, timeout_ms=1000.0, interleave=0) -> ct_measure_opts:
    return ct_measure_opts(int(warmup), int(repeats), int(launches), int(batch), float(timeout_ms),
                           int(interleave))


def opts_from_protocol(p, batch=16, interleave=0) -> ct_measure_opts:
    return make_opts(p.warmup, p.repeats, p.launches, batch, p.timeout_ms, interleave)


def mask_array(mask) -> ctypes.Array:
    arr = (c_u32 * MASK_WORDS)()
    for i, v in enumerate(mask):
        arr[i] = int(v)
    return arr


# ---------------------------------------------------------------- entry points
def ct_init(device: int = 0) -> None:
    _check(lib().ct_init(device))


def ct_num_cus() -> int:
    return _check(lib().ct_num_cus())


def ct_shutdown() -> None:
    lib().ct_shutdown()


def ct_stream_count() -> int:
    return _check(lib().ct_stream_count())


def ct_last_error() -> str:
    return lib().ct_last_error().decode(errors="replace")


def ct_build_cu_mask(num_cus: int, fraction: float, slot: int) -> np.ndarray:
    m = np.zeros(MASK_WORDS, dtype=np.uint32)
    _check(lib().ct_build_cu_mask(num_cus, fraction, slot, _arr(m, c_u32), MASK_WORDS))
    return m


def ct_cu_mask(fraction: float, slot: int = 0) -> np.ndarray:
    m = np.zeros(MASK_WORDS, dtype=np.uint32)
    _check(lib().ct_cu_mask(fraction, slot, _arr(m, c_u32), MASK_WORDS))
    return m


def ct_grid_info(family: int):
    nk, gs = c_i32(), c_i64()
    _check(lib().ct_grid_info(family, ctypes.byref(nk), ctypes.byref(gs)))
    return nk.value, gs.value


def ct_grid_size(op, family: int) -> int:
    """Number of schedules of `family` the validator accepts for op."""
    o = make_op(op)
    n = c_i64()
    _check(lib().ct_grid_size(ctypes.byref(o), family, ctypes.byref(n)))
    return n.value


def ct_set_reference(op, y_ref_host: Optional[np.ndarray]) -> None:
    """Register op's exact output (fp64, op's output layout) for later
    measurements; None removes it."""
    o = make_op(op)
    if y_ref_host is None:
        _check(lib().ct_set_reference(ctypes.byref(o), None))
        return
    ref = np.ascontiguousarray(y_ref_host, dtype=np.float64)
    _check(lib().ct_set_reference(ctypes.byref(o), _arr(ref, c_f64)))


def ct_knob_values(family: int, knob: int) -> List[int]:
    vals = (c_i32 * 32)()
    cnt = c_i32()
    _check(lib().ct_knob_values(family, knob, vals, 32, ctypes.byref(cnt)))
    return [vals[i] for i in range(cnt.value)]


def ct_grid_decode(family: int, index: int) -> ct_schedule:
    s = ct_schedule()
    _check(lib().ct_grid_decode(family, index, ctypes.byref(s)))
    return s


def ct_grid_encode(s: ct_schedule) -> int:
    idx = c_i64()
    _check(lib().ct_grid_encode(ctypes.byref(s), ctypes.byref(idx)))
    return idx.value


def ct_validate(op, s: ct_schedule) -> int:
    """0 if valid, S_INVALID (1) if rejected; raises on malformed input."""
    o = make_op(op)
    return _check(lib().ct_validate(ctypes.byref(o), ctypes.byref(s)))


def ct_launch_shape(op, s: ct_schedule):
    o = make_op(op)
    lds, th, ker = c_i32(), c_i32(), c_i32()
    blocks = c_i64()
    _check(lib().ct_launch_shape(ctypes.byref(o), ctypes.byref(s), ctypes.byref(lds), ctypes.byref(th),
                                 ctypes.byref(blocks), ctypes.byref(ker)))
    return {"lds_bytes": lds.value, "threads": th.value, "blocks": blocks.value, "kernels": ker.value}


def ct_kernel_name(op, s: ct_schedule) -> str:
    o = make_op(op)
    buf = ctypes.create_string_buffer(256)
    _check(lib().ct_kernel_name(ctypes.byref(o), ctypes.byref(s), buf, 256))
    return buf.value.decode()


def ct_valid_space(op) -> ctypes.Array:
    o = make_op(op)
    cnt = c_i64()
    _check(lib().ct_valid_space(ctypes.byref(o), None, 0, ctypes.byref(cnt)))
    arr = (ct_schedule * max(cnt.value, 1))()
    _check(lib().ct_valid_space(ctypes.byref(o), arr, cnt.value, ctypes.byref(cnt)))
    return arr[:cnt.value]


def ct_sample(op, seed: int, config_id: int, layer_id: int, n: int) -> List[ct_schedule]:
    o = make_op(op)
    arr = (ct_schedule * max(n, 1))()
    got = c_i32()
    _check(lib().ct_sample(ctypes.byref(o), seed, config_id, layer_id, n, arr, ctypes.byref(got)))
    return [arr[i] for i in range(got.value)]


def ct_sample_uniform(op, seed: int, config_id: int, layer_id: int, n: int) -> List[ct_schedule]:
    o = make_op(op)
    arr = (ct_schedule * max(n, 1))()
    got = c_i32()
    _check(lib().ct_sample_uniform(ctypes.byref(o), seed, config_id, layer_id, n, arr, ctypes.byref(got)))
    return [arr[i] for i in range(got.value)]


def conv2d_run(op, s: ct_schedule, x, w, y, cu_mask=None) -> None:
    o = make_op(op)
    m = mask_array(cu_mask) if cu_mask is not None else None
    _check(lib().conv2d_run(ctypes.byref(o), ctypes.byref(s), _ptr(x), _ptr(w), _ptr(y), m,
                            MASK_WORDS if m is not None else 0))


SCRATCH_FLOATS = 1 << 24


def conv2d_run_noalloc(op, s: ct_schedule, x, w, y, stream: int = 0) -> None:
    """conv2d_run without any allocation: enqueued on `stream` (a raw HIP
    stream handle, 0 = the null stream), returns without waiting."""
    o = make_op(op)
    _check(lib().conv2d_run_noalloc(ctypes.byref(o), ctypes.byref(s), _ptr(x), _ptr(w), _ptr(y),
                                    ctypes.c_void_p(stream) if stream else None))


def measure_candidates(op, scheds: Sequence, cu_fraction: float, opts: ct_measure_opts, x, w, y):
    o = make_op(op)
    arr = schedule_array(scheds)
    n = len(scheds)
    lat = np.zeros(max(n, 1), dtype=np.float32)
    st = np.zeros(max(n, 1), dtype=np.int32)
    _check(lib().measure_candidates(ctypes.byref(o), arr, n, cu_fraction, ctypes.byref(opts), _ptr(x), _ptr(w),
                                    _ptr(y), _arr(lat, c_f32), _arr(st, c_i32)))
    return lat[:n], st[:n]


def measure_candidates_mask(op, scheds: Sequence, cu_mask, opts: ct_measure_opts, x, w, y, y_ref=None,
                            tol: float = 0.0, want_repeats: bool = False):
    o = make_op(op)
    arr = schedule_array(scheds)
    n = len(scheds)
    lat = np.zeros(max(n, 1), dtype=np.float32)
    st = np.zeros(max(n, 1), dtype=np.int32)
    rep = np.zeros(max(n, 1) * opts.repeats, dtype=np.float32) if want_repeats else None
    v = ct_verify(_ptr(y_ref), float(tol)) if y_ref is not None else None
    m = mask_array(cu_mask) if cu_mask is not None else None
    _check(lib().measure_candidates_mask(ctypes.byref(o), arr, n, m, MASK_WORDS if m is not None else 0,
                                         ctypes.byref(opts), ctypes.byref(v) if v is not None else None,
                                         _ptr(x), _ptr(w), _ptr(y), _arr(lat, c_f32), _arr(st, c_i32),
                                         _arr(rep, c_f32) if rep is not None else None))
    if want_repeats:
        return lat[:n], st[:n], rep[:n * opts.repeats].reshape(n, opts.repeats)
    return lat[:n], st[:n]


def ct_top_t(lat: np.ndarray, status: np.ndarray, t: int) -> np.ndarray:
    lat = np.ascontiguousarray(lat, dtype=np.float32)
    status = np.ascontiguousarray(status, dtype=np.int32)
    top = np.zeros(max(t, 1), dtype=np.int32)
    cnt = c_i32()
    _check(lib().ct_top_t(_arr(lat, c_f32), _arr(status, c_i32), len(lat), t, _arr(top, c_i32), ctypes.byref(cnt)))
    return top[:cnt.value]


def ct_select_winner(lat: np.ndarray, pos: np.ndarray, eps: float) -> int:
    lat = np.ascontiguousarray(lat, dtype=np.float32)
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    wi = c_i32()
    _check(lib().ct_select_winner(_arr(lat, c_f32), _arr(pos, c_i32), len(lat), eps, ctypes.byref(wi)))
    return wi.value


def ct_tune_clients(clients: ctypes.Array, opts1: ct_measure_opts, opts2: ct_measure_opts, eps: float) -> None:
    _check(lib().ct_tune_clients(clients, len(clients), ctypes.byref(opts1), ctypes.byref(opts2), eps))


def ct_tune_shared(clients: ctypes.Array, jobs: ctypes.Array, opts1: ct_measure_opts, opts2: ct_measure_opts,
                   eps: float) -> np.ndarray:
    """Run the clients on one shared job queue; returns the client index per job."""
    owner = np.full(max(len(jobs), 1), -1, dtype=np.int32)
    _check(lib().ct_tune_shared(clients, len(clients), jobs, len(jobs), ctypes.byref(opts1), ctypes.byref(opts2),
                                eps, _arr(owner, c_i32)))
    return owner[:len(jobs)]


def ct_throughput(clients: ctypes.Array) -> float:
    """Aggregate candidates/s of clients that have run (sum over the makespan)."""
    v = c_f64()
    _check(lib().ct_throughput(clients, len(clients), ctypes.byref(v)))
    return v.value


def ct_tune_split(job: ct_tune_job, masks: Sequence, y_slots: Sequence, opts1: ct_measure_opts,
                  opts2: ct_measure_opts, eps: float) -> float:
    """Screen one job's candidates on len(masks) CU slots at once, merge, then
    re-measure and select on slot 0; returns the screening seconds."""
    k = len(masks)
    mk = np.ascontiguousarray(np.array(masks, dtype=np.uint32).reshape(k, MASK_WORDS))
    ys = (ctypes.c_void_p * k)(*[_ptr(y) for y in y_slots])
    sec = c_f64()
    _check(lib().ct_tune_split(ctypes.byref(job), _arr(mk, c_u32), k, MASK_WORDS, ys, ctypes.byref(opts1),
                               ctypes.byref(opts2), eps, ctypes.byref(sec)))
    return sec.value


def ct_test_run_clients(clients: ctypes.Array, jobs: ctypes.Array, hooks: ct_test_hooks) -> np.ndarray:
    """The client machinery with the library's stand-in measurement (host only);
    returns the client index per job. Raises CtError with the call's code."""
    owner = np.full(max(len(jobs), 1), -1, dtype=np.int32)
    _check(lib().ct_test_run_clients(clients, len(clients), jobs, len(jobs), ctypes.byref(hooks),
                                     _arr(owner, c_i32)))
    return owner[:len(jobs)]


def ct_test_watchdog(runs: Sequence[int], done_at_s: Sequence[float], run_limit_s: float, slack_s: float,
                     drain_cap_s: float):
    """The timeout watchdog on a simulated stream: (expired event or -1, drained)."""
    r = np.ascontiguousarray(runs, dtype=np.int32)
    d = np.ascontiguousarray(done_at_s, dtype=np.float64)
    ex, dr = c_i32(), c_i32()
    _check(lib().ct_test_watchdog(len(r), _arr(r, c_i32), _arr(d, c_f64), run_limit_s, slack_s, drain_cap_s,
                                  ctypes.byref(ex), ctypes.byref(dr)))
    return ex.value, bool(dr.value)


def ct_test_xcd_band(tiles: int) -> np.ndarray:
    """Tile of each block under the bf16 family's XCD-band renumbering."""
    out = np.zeros(tiles, dtype=np.int32)
    _check(lib().ct_test_xcd_band(tiles, _arr(out, c_i32)))
    return out


def ct_cross_eval(op, scheds: Sequence, masks: Sequence, opts: ct_measure_opts, x, w, y) -> np.ndarray:
    o = make_op(op)
    arr = schedule_array(scheds)
    mk = np.ascontiguousarray(np.array(masks, dtype=np.uint32).reshape(len(masks), MASK_WORDS))
    M = np.zeros(len(scheds) * len(masks), dtype=np.float32)
    _check(lib().ct_cross_eval(ctypes.byref(o), arr, len(scheds), _arr(mk, c_u32), len(masks), MASK_WORDS,
                               ctypes.byref(opts), _ptr(x), _ptr(w), _ptr(y), _arr(M, c_f32)))
    return M.reshape(len(scheds), len(masks))


def make_search_opts(seed=0, batch=16, budget=256, patience=0, sa_chains=32, sa_steps=100, explore=0.25,
                     eps=0.01, sa_temp=0.5, cus=0) -> ct_search_opts:
    return ct_search_opts(int(seed), int(batch), int(budget), int(patience), int(sa_chains), int(sa_steps),
                          float(explore), float(eps), float(sa_temp), int(cus))


def ct_search_propose(op, measured: Sequence, lat_us, status, so: ct_search_opts, round_: int,
                      cap: Optional[int] = None) -> List[ct_schedule]:
    n = len(measured)
    cap = so.batch if cap is None else cap
    arr = schedule_array(measured) if n else None
    lat = np.ascontiguousarray(lat_us, dtype=np.float32) if n else np.zeros(1, np.float32)
    st = np.ascontiguousarray(status, dtype=np.int32) if n else np.zeros(1, np.int32)
    out = (ct_schedule * max(cap, 1))()
    cnt = c_i32()
    o = make_op(op)
    _check(lib().ct_search_propose(ctypes.byref(o), arr, _arr(lat, c_f32), _arr(st, c_i32), n, ctypes.byref(so),
                                   int(round_), out, int(cap), ctypes.byref(cnt)))
    return [out[i] for i in range(cnt.value)]


def ct_search(op, so: ct_search_opts, cu_mask, stage1: ct_measure_opts, stage2: ct_measure_opts, top_t: int,
              eps: float, x, w, y):
    """Guided search on one mask: (measured schedules, stage-1 latencies,
    statuses, result fields as a dict)."""
    n = so.budget
    meas = (ct_schedule * n)()
    lat = np.zeros(n, dtype=np.float32)
    st = np.zeros(n, dtype=np.int32)
    res = ct_search_result()
    o = make_op(op)
    m = mask_array(cu_mask) if cu_mask is not None else None
    _check(lib().ct_search(ctypes.byref(o), ctypes.byref(so), m, MASK_WORDS if m is not None else 0,
                           ctypes.byref(stage1), ctypes.byref(stage2), int(top_t), float(eps), _ptr(x), _ptr(w),
                           _ptr(y), meas, _arr(lat, c_f32), _arr(st, c_i32), ctypes.byref(res)))
    k = res.n_measured
    info = {f: getattr(res, f) for f, _ in ct_search_result._fields_ if f != "pad_"}
    return [meas[i] for i in range(k)], lat[:k], st[:k], info


def ct_probe_cus(cu_mask, blocks: int = 4096) -> np.ndarray:
    out = np.zeros(1024, dtype=np.int32)
    cnt = c_i32()
    m = mask_array(cu_mask) if cu_mask is not None else None
    _check(lib().ct_probe_cus(m, MASK_WORDS if m is not None else 0, blocks, _arr(out, c_i32), 1024,
                              ctypes.byref(cnt)))
    return out[:min(cnt.value, 1024)]


def ct_probe_empty(cu_mask, blocks: int, opts: ct_measure_opts) -> float:
    us = c_f32()
    m = mask_array(cu_mask) if cu_mask is not None else None
    _check(lib().ct_probe_empty(m, MASK_WORDS if m is not None else 0, blocks, ctypes.byref(opts),
                                ctypes.byref(us)))
    return us.value


def ct_probe_copy(cu_mask, src, dst, nbytes: int, opts: ct_measure_opts) -> float:
    g = c_f32()
    m = mask_array(cu_mask) if cu_mask is not None else None
    _check(lib().ct_probe_copy(m, MASK_WORDS if m is not None else 0, _ptr(src), _ptr(dst), nbytes,
                               ctypes.byref(opts), ctypes.byref(g)))
    return g.value


def header_functions(header_path: Optional[str] = None) -> List[str]:
    """Names of the functions declared in include/convtune.h (for export checks)."""
    import re
    path = header_path or os.path.join(os.path.dirname(os.path.dirname(LIB_PATH)), "include", "convtune.h")
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?(?:int|void|char)\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))
