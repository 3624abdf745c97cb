"""Stored expected values under tests/golden/.

* conv2d_by_hand.json: convolutions worked by hand from the operator's
  definition (each case names the arithmetic it follows). The oracle must
  reproduce them exactly; the GPU test runs every applicable kernel family
  on them through the C ABI (small integers: the results are exact).
* host_rules_oracle.json: the oracle's seeded sample on fixed family sizes
  and its CU masks, written by tests/golden/make_golden.py; the masks are
  also checked against their rule by hand.
"""
import json
import os
import random

import numpy as np
import pytest

import oracle
import oracle.host_rules as HR

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(HERE, name)) as fh:
        return json.load(fh)


HAND = _load("conv2d_by_hand.json")["cases"]


@pytest.mark.parametrize("case", HAND, ids=lambda c: c["name"])
def test_oracle_reproduces_hand_worked_convolutions(case):
    x = np.array(case["x"], dtype=np.float64)
    w = np.array(case["w"], dtype=np.float64)
    y = oracle.conv2d(x, w, tuple(case["stride"]), tuple(case["pad"]), tuple(case["dil"]), case["groups"])
    assert np.array_equal(y, np.array(case["y"], dtype=np.float64)), case["cite"]


def test_oracle_sampler_and_masks_match_stored_values():
    g = _load("host_rules_oracle.json")
    for s in g["samples"]:
        got = HR.sample_positions(s["families"], s["sizes"], s["n"], s["seed"], s["config_id"], s["layer_id"])
        assert got == s["positions"]
        # a valid sample: distinct positions inside the valid list, the family
        # quotas met
        assert len(set(got)) == len(got) == min(s["n"], sum(s["sizes"]))
        assert all(0 <= p < sum(s["sizes"]) for p in got)
    for m in g["cu_masks"]:
        assert HR.cu_mask(256, m["fraction"], m["slot"]) == m["words"]
    # by hand: an eighth of 256 CUs is 32, so slot 1 is CUs 32..63 = word 1
    eighth = [m for m in g["cu_masks"] if m["fraction"] == 0.125 and m["slot"] == 1][0]
    assert eighth["words"] == [0, 0xFFFFFFFF, 0, 0, 0, 0, 0, 0]
    full = [m for m in g["cu_masks"] if m["fraction"] == 1.0][0]
    assert full["words"] == [0xFFFFFFFF] * 8


@pytest.mark.gpu
@pytest.mark.parametrize("case", HAND, ids=lambda c: c["name"])
def test_hand_worked_convolutions_on_every_family(case):
    import torch
    from gpu_util import device_ready, note, sched_str
    from paper_2008_03602_amd import _lib as L, workloads as W

    device_ready()
    x = np.array(case["x"], dtype=np.float32)
    w = np.array(case["w"], dtype=np.float32)
    n, c, h, wd = x.shape
    k, _, r, s = w.shape
    op = W.Op(case["name"], n, c, h, wd, k, r, s, case["stride"][0], case["stride"][1], case["pad"][0],
              case["pad"][1], case["dil"][0], case["dil"][1], case["groups"])
    want = np.array(case["y"], dtype=np.float32)
    xd = torch.from_numpy(x).cuda()
    wdv = torch.from_numpy(w).cuda()
    yd = torch.empty(op.y_shape(), dtype=torch.float32, device="cuda")
    space = L.ct_valid_space(op)
    fams = sorted({int(sc.family) for sc in space})
    if not fams:
        pytest.skip("no schedule of any family is valid for this shape")
    rng = random.Random(3)
    for f in fams:
        pool = [sc for sc in space if sc.family == f]
        for sc in rng.sample(pool, min(6, len(pool))):
            tag = "%s %s" % (case["name"], sched_str(sc))
            note(tag)
            yd.fill_(float("nan"))
            L.conv2d_run(op, sc, xd, wdv, yd)
            assert np.array_equal(yd.cpu().numpy(), want), tag
