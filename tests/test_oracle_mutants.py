"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a temporary copy of the C oracle (on the CPU,
never in the committed file), builds it, and checks that the pin battery --
exact scatter-form brute force, the delta filter and the NHWC/NCHW
consistency -- rejects it.
"""
import os
import random
import subprocess

import numpy as np
import pytest

import oracle
from oracle.brute import conv2d_scatter

SRC = os.path.join(os.path.dirname(oracle.__file__), "conv2d_ref.c")

MUTANTS = {
    "dropped_pad_term": ("p * sh - ph + r * dh", "p * sh + r * dh"),
    "wrong_sign_pad": ("q * sw - pw + t * dw", "q * sw + pw + t * dw"),
    "transposed_filter_taps": ("w_at(layout, k, c, r, t, Cg, R, S)", "w_at(layout, k, c, t, r, Cg, S, R)"),
    "group_offset_dropped": ("const int64_t c0 = (k / Kg) * Cg;", "const int64_t c0 = 0 * Kg;"),
    "output_size_floor_off": ("return span / stride + 1;", "return (span + stride - 1) / stride + 1;"),
    "dilation_ignored": ("+ r * dh;", "+ r;"),
    "nhwc_h_w_swapped": ("return ((n * H + h) * W + w) * C + c;", "return ((n * W + w) * H + h) * C + c;"),
    "filter_flipped": ("const double wv = w[w_at(layout, k, c, r, t, Cg, R, S)];",
                       "const double wv = w[w_at(layout, k, c, R - 1 - r, S - 1 - t, Cg, R, S)];"),
    "stride_w_uses_h": ("const int64_t wi = q * sw - pw + t * dw;", "const int64_t wi = q * sh - pw + t * dw;"),
}


def _battery(lib):
    """True when every pin holds for the oracle library ``lib``."""
    rng = random.Random(99)
    cases = [(1, 3, 5, 6, 3, 3, 2, (1, 2), (1, 0), (1, 1), 1),
             (2, 2, 6, 5, 4, 2, 3, (2, 1), (2, 1), (2, 1), 2),
             (1, 3, 6, 6, 3, 3, 3, (1, 1), (1, 1), (1, 2), 3),
             (1, 2, 4, 7, 2, 1, 3, (1, 2), (0, 2), (1, 1), 1),
             (1, 1, 7, 5, 2, 3, 1, (2, 2), (0, 0), (1, 1), 1)]
    for (N, C, H, Wd, K, R, S, st, pd, dl, g) in cases:
        x = np.array([rng.randint(-8, 8) for _ in range(N * C * H * Wd)], float).reshape(N, C, H, Wd)
        w = np.array([rng.randint(-8, 8) for _ in range(K * (C // g) * R * S)], float).reshape(K, C // g, R, S)
        ref = np.array(conv2d_scatter(x.tolist(), w.tolist(), N, C, H, Wd, K, R, S, st, pd, dl, g), float)
        try:
            y = oracle.conv2d(x, w, st, pd, dl, g, lib=lib)
        except ValueError:
            return False
        if y.shape != ref.shape or not np.array_equal(y, ref):
            return False
        y2 = oracle.conv2d(x.transpose(0, 2, 3, 1), w.transpose(0, 2, 3, 1), st, pd, dl, g,
                           layout="nhwc", lib=lib)
        if not np.array_equal(y2, ref.transpose(0, 2, 3, 1)):
            return False
    x = np.arange(2 * 3 * 7 * 8, dtype=float).reshape(2, 3, 7, 8)
    w = np.zeros((3, 3, 3, 3))
    for k in range(3):
        w[k, k, 1, 1] = 1.0
    y = oracle.conv2d(x, w, (1, 1), (1, 1), lib=lib)
    return y.shape == x.shape and np.array_equal(y, x)


def test_battery_accepts_the_real_oracle():
    assert _battery(None)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_battery_rejects_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, "mutation anchor missing: " + old
    mutated = src.replace(old, new)
    cfile = tmp_path / "mut.c"
    cfile.write_text(mutated)
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O1", "-fPIC", "-shared", "-std=c99", "-o", str(so), str(cfile), "-lm"])
    lib = oracle.load_library(str(so))
    assert not _battery(lib), "pins did not catch mutant " + name
