"""GPU parity of code paths that a random sample of schedules may miss, against
the fp64 oracle, through the C ABI:

* fp32 MFMA schedules with four loader waves (stages 3), with 1, 2 and 4
  reduction groups and with one chunk or several;
* direct schedules without LDS whose chunks end in an odd channel count while
  two channels go per step (UNR 2), for 3x3 and 1x1 filters, and the
  register-bound instances that take one channel per step;
* the direct generic-filter path (7x7, 5x3 and dilated filters), whose filter
  rows do not divide into its tap groups;
* fp32 MFMA schedules whose 16-pixel MFMA columns span two 8-pixel halo rows
  16 words apart, where the halo's channel pitch is 8 (mod 32) instead of 16.
Every case also runs on integer inputs, where any summation order is exact.
"""
import random

import numpy as np
import pytest

from paper_2008_03602_amd import _lib as L, workloads as W
from gpu_util import check_close, device_ready, make_inputs, note, reference, sched_str, to_device

pytestmark = pytest.mark.gpu

# knob positions (the schedule's documented order)
F4_WS, F4_TPW, F4_CPC, F4_STAGES = 5, 6, 7, 8
D_LDS, D_CT, D_UNR, D_MK, D_MW = 5, 6, 8, 3, 4


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _run(op, scheds, seed):
    for dist, exact in (("uniform", False), ("int", True)):
        x, w = make_inputs(op, dist, seed=seed, int_range=2)
        ref, a = reference(op, x, w)
        xd, wd, yd = to_device(op, x, w)
        for s in scheds:
            tag = "%s %s %s" % (op.name, dist, sched_str(s))
            note(tag)
            yd.fill_(float("nan"))
            L.conv2d_run(op, s, xd, wd, yd)
            y = yd.cpu().numpy()
            if exact:
                assert np.array_equal(y.astype(np.float64), ref), tag + ": not bit-exact on integer inputs"
            else:
                check_close(op, y, ref, a, tag, split=W.split_of(s))


def _pick(pool, key, per_key, rng):
    """per_key schedules for every value of key(s) found in pool."""
    out = []
    for v in sorted({key(s) for s in pool}):
        grp = [s for s in pool if key(s) == v]
        out += rng.sample(grp, min(per_key, len(grp)))
    return out


LOADER_OPS = [
    W.conv("ld_vec3x3", 1, 24, 20, 40, 3, 1),      # 16-byte copies, ragged K
    W.conv("ld_odd3x3", 1, 5, 13, 11, 3, 1),       # 4-byte copies, C = 5
    W.conv("ld_pw", 2, 32, 12, 20, 1, 1, 0),
    W.conv("ld_deep", 1, 64, 14, 48, 3, 1),        # several chunks
]


@pytest.mark.parametrize("op", LOADER_OPS, ids=lambda o: o.name)
def test_loader_wave_schedules_match_oracle(op):
    pool = [s for s in L.ct_valid_space(op) if s.family == W.FAM_IGEMM_F32 and s.knob[F4_STAGES] == 3]
    assert pool, "no loader schedule is valid on " + op.name
    rng = random.Random(3)
    # every reduction-group count, and one chunk as well as several
    picks = _pick(pool, lambda s: (s.knob[F4_WS], s.knob[F4_CPC] >= op.c), 2, rng)
    assert {s.knob[F4_WS] for s in picks} >= {1, 2}
    _run(op, picks, seed=21)


UNR_OPS = [
    W.conv("unr_3x3", 1, 7, 11, 12, 3, 1),         # C = 7: chunks of 2 and 4 end odd
    W.conv("unr_3x3s2", 1, 9, 14, 10, 3, 2),
    W.conv("unr_1x1", 2, 13, 9, 16, 1, 1, 0),
]


@pytest.mark.parametrize("op", UNR_OPS, ids=lambda o: o.name)
def test_direct_two_channel_steps_with_odd_tails_match_oracle(op):
    pool = [s for s in L.ct_valid_space(op)
            if s.family == W.FAM_DIRECT_F32 and s.knob[D_LDS] == 0 and s.knob[D_UNR] == 2
            and (min(s.knob[D_CT], op.c) % 2 == 1 or op.c % s.knob[D_CT] % 2 == 1)]
    assert pool
    rng = random.Random(5)
    # small register tiles (two channels per step) and large ones (one)
    picks = _pick(pool, lambda s: s.knob[D_MK] * s.knob[D_MW] >= 8, 4, rng)
    _run(op, picks, seed=22)


GENERIC_OPS = [
    W.conv("gen_7x7s2", 1, 3, 23, 8, 7, 2, 3),
    W.Op("gen_5x3", 1, 4, 12, 13, 6, 5, 3, 1, 1, 2, 1, 1, 1, 1, 0, 0),
    W.Op("gen_dil", 1, 4, 11, 11, 6, 3, 3, 1, 1, 2, 2, 2, 2, 1, 0, 0),
]


@pytest.mark.parametrize("op", GENERIC_OPS, ids=lambda o: o.name)
def test_direct_generic_filter_tap_groups_match_oracle(op):
    pool = [s for s in L.ct_valid_space(op) if s.family == W.FAM_DIRECT_F32 and s.knob[D_LDS] == 0]
    assert pool
    rng = random.Random(7)
    picks = _pick(pool, lambda s: (s.knob[D_UNR], s.knob[D_MK] * s.knob[D_MW] >= 8), 2, rng)
    _run(op, picks, seed=23)


TWO_ROW_OPS = [
    W.conv("tr_3x3", 2, 12, 20, 24, 3, 1),                            # 3x3 fixed-filter path
    W.Op("tr_5x5", 1, 6, 16, 16, 10, 5, 5, 1, 1, 2, 2, 1, 1, 1, 0, 0),  # generic path, rows of 16
]


@pytest.mark.parametrize("op", TWO_ROW_OPS, ids=lambda o: o.name)
def test_two_row_halo_pitch_schedules_match_oracle(op):
    # 16x16 MFMAs over 8-pixel tiles at stride 1 with 16-byte halo rows of 16
    # words: every such schedule takes the two-row channel pitch
    pool = [s for s in L.ct_valid_space(op) if s.family == W.FAM_IGEMM_F32 and s.knob[0] == 16
            and s.knob[F4_TPW] == 8]
    assert pool
    rng = random.Random(11)
    picks = _pick(pool, lambda s: (s.knob[F4_STAGES], s.knob[F4_WS]), 1, rng)
    assert {s.knob[F4_STAGES] for s in picks} == {1, 2, 3}
    _run(op, picks, seed=24)
