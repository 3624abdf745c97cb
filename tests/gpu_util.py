"""Helpers of the GPU tests: device buffers, oracle references, error checks."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2008_03602_amd import _lib as L, synth, workloads as W

U = 2.0 ** -24  # unit roundoff of fp32


def note(msg: str) -> None:
    """Say which case is about to touch the GPU (flushed, so a crash still names it)."""
    print("[gpu-case] " + msg, flush=True)
    sys.stdout.flush()


def device_ready() -> None:
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    L.ct_init(0)


def make_inputs(op: W.Op, dist: str, seed: int = 0, config_id: int = 0, layer_id: int = 0,
                int_range: int = 2):
    bf16 = op.dtype == W.DT_BF16
    x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), dist, seed, config_id, layer_id, bf16=bf16,
                             int_range=int_range)
    return x, w


def reference(op: W.Op, x: np.ndarray, w: np.ndarray, threads: int = 8):
    """fp64 oracle output and |x|*|w| bound, in the op's output layout."""
    lay = "nchw" if op.layout == W.LAYOUT_NCHW else "nhwc"
    y, a = oracle.conv2d(x, w, (op.stride_h, op.stride_w), (op.pad_h, op.pad_w), (op.dil_h, op.dil_w),
                         op.groups, layout=lay, threads=threads, with_abs=True)
    return y, a


def to_device(op: W.Op, x: np.ndarray, w: np.ndarray):
    dev = torch.device("cuda:0")
    if op.dtype == W.DT_BF16:
        xd = torch.from_numpy(synth.bf16_bits(x).view(np.int16).copy()).to(dev)
        wd = torch.from_numpy(synth.bf16_bits(w).view(np.int16).copy()).to(dev)
    else:
        xd = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev)
        wd = torch.from_numpy(np.ascontiguousarray(w, dtype=np.float32)).to(dev)
    yd = torch.full(op.y_shape(), float("nan"), dtype=torch.float32, device=dev)
    return xd, wd, yd


def reduction_length(op: W.Op) -> int:
    return op.cg * op.r * op.s


def check_close(op: W.Op, y: np.ndarray, ref: np.ndarray, a: np.ndarray, what: str, split: int = 1):
    """Spec tolerance (infinity-norm relative) and the element-wise fp32 summation bound."""
    tol = 2e-2 if op.dtype == W.DT_BF16 else 1e-4
    assert y.shape == ref.shape, what
    assert np.all(np.isfinite(y)), what + ": non-finite output"
    err = np.abs(y.astype(np.float64) - ref)
    scale = max(float(np.max(np.abs(ref))), 1e-30)
    rel = float(np.max(err)) / scale
    assert rel <= tol, "%s: relative error %.3e > %.1e" % (what, rel, tol)
    # any summation order of n fp32 terms errs by at most about n*u*sum|terms|; the
    # final rounding of y and the split partial sums add a few more units
    n = reduction_length(op) + split + 2
    bound = n * U * a + 1e-30
    worst = float(np.max(err / bound))
    assert worst <= 1.0, "%s: error exceeds the fp32 summation bound by %.2fx" % (what, worst)
    return rel


def sched_str(s) -> str:
    t = L.schedule_tuple(s)
    nk, _ = L.ct_grid_info(t[0])
    return "%s%s" % (W.FAMILY_NAMES[t[0]], list(t[1:1 + nk]))
