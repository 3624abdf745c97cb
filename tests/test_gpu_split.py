"""Schedules that split their reduction, through the C ABI.

Schedules that split their reduction 2 to 8 ways, from every family with the
knob, run back to back on one stream's workspace, with new inputs each round
and in a new order: a partial sum left behind by another launch or another
split count would show up here as a wrong output against the fp64 oracle.
Then the same schedules run under the timing protocol (dozens of launches
each, outputs verified on the device) on a quarter share, and afterwards
every rerun gives the same bits (the partials are added in split order).
"""
import random

import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, workloads as W
from gpu_util import check_close, device_ready, make_inputs, note, reference, sched_str, to_device

pytestmark = pytest.mark.gpu

OPS = [
    W.conv("sp3x3", 1, 64, 14, 48, 3, 1),  # direct and fp32 MFMA, splits of 2, 4 and 8
    W.conv("sp_pw_bf", 2, 128, 7, 40, 1, 1, 0, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC),
]


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _split_scheds(op, per_split=2, seed=0):
    """per_split schedules for every (family, split > 1) the op's space holds."""
    space = [s for s in L.ct_valid_space(op) if W.split_of(s) > 1]
    rng = random.Random(seed)
    out = []
    for fam in sorted({int(s.family) for s in space}):
        for sp in sorted({W.split_of(s) for s in space if s.family == fam}):
            pool = [s for s in space if s.family == fam and W.split_of(s) == sp]
            out += rng.sample(pool, min(per_split, len(pool)))
    return out


def _tol(op):
    return 2e-2 if op.dtype == W.DT_BF16 else 1e-4


@pytest.mark.parametrize("op", OPS, ids=lambda o: o.name)
def test_split_schedules_back_to_back_match_oracle(op):
    scheds = _split_scheds(op)
    assert len({W.split_of(s) for s in scheds}) >= 2
    for rnd in range(2):
        x, w = make_inputs(op, "uniform", seed=100 + rnd)
        ref, a = reference(op, x, w)
        xd, wd, yd = to_device(op, x, w)
        for s in (scheds if rnd == 0 else scheds[::-1]):
            tag = "%s round %d %s" % (op.name, rnd, sched_str(s))
            note(tag)
            yd.fill_(float("nan"))
            L.conv2d_run(op, s, xd, wd, yd)
            check_close(op, yd.cpu().numpy(), ref, a, tag, split=W.split_of(s))


@pytest.mark.parametrize("op", OPS, ids=lambda o: o.name)
def test_split_under_timing_then_reruns_identical(op):
    scheds = _split_scheds(op, per_split=1, seed=1)
    x, w = make_inputs(op, "normal", seed=7)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    note("%s: timing %d split schedules on a quarter share" % (op.name, len(scheds)))
    yref = torch.from_numpy(ref.astype(np.float32)).cuda()
    lat, st = L.measure_candidates_mask(op, scheds, L.ct_cu_mask(0.25, 0), L.make_opts(2, 5, 10), xd, wd, yd,
                                        y_ref=yref, tol=_tol(op))
    assert list(st) == [L.S_OK] * len(scheds), [L.STATUS_NAMES[int(v)] for v in st]
    assert np.all(np.isfinite(lat))
    for s in scheds:
        tag = "%s rerun %s" % (op.name, sched_str(s))
        note(tag)
        outs = []
        for _ in range(3):
            yd.fill_(float("nan"))
            L.conv2d_run(op, s, xd, wd, yd)
            outs.append(yd.cpu().numpy())
        check_close(op, outs[0], ref, a, tag, split=W.split_of(s))
        assert all(np.array_equal(outs[0], o) for o in outs[1:]), tag + ": reruns differ"
