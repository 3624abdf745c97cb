"""GPU tests of CU masks, the timing protocol, verification and tuning clients."""
import numpy as np
import pytest
import torch

import oracle.host_rules as HR
from paper_2008_03602_amd import _lib as L, workloads as W
from gpu_util import device_ready, make_inputs, note, reference, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _xcc(ids):
    return np.asarray(ids) >> 12


def test_full_mask_reaches_every_cu():
    note("probe full mask")
    n = L.ct_num_cus()
    ids = L.ct_probe_cus(None, blocks=16 * n)
    assert len(ids) == n
    assert len(np.unique(_xcc(ids))) == 8


@pytest.mark.parametrize("fraction", [0.125, 0.25, 0.5])
def test_slots_are_disjoint_and_balanced_over_xcds(fraction):
    n = L.ct_num_cus()
    slots = int(round(1 / fraction))
    seen = []
    for j in range(slots):
        m = L.ct_cu_mask(fraction, j)
        note("probe fraction %.3f slot %d" % (fraction, j))
        ids = L.ct_probe_cus(m, blocks=16 * n)
        want = int(round(n * fraction))
        assert len(ids) == want, "slot %d saw %d CUs, mask has %d" % (j, len(ids), want)
        per_xcd = np.bincount(_xcc(ids), minlength=8)
        assert per_xcd.min() == per_xcd.max() == want // 8, per_xcd
        seen.append(set(ids.tolist()))
    for a in range(slots):
        for b in range(a + 1, slots):
            assert not (seen[a] & seen[b])


def test_measure_protocol_and_median():
    op = W.config(1).ops[0]
    x, w = make_inputs(op, "uniform", config_id=1)
    xd, wd, yd = to_device(op, x, w)
    scheds = L.ct_sample(op, 0, 1, 0, 8)
    opts = L.make_opts(warmup=1, repeats=5, launches=4, batch=4)
    note("measure 8 candidates config1")
    lat, st, rep = L.measure_candidates_mask(op, scheds, L.ct_cu_mask(1.0, 0), opts, xd, wd, yd,
                                             want_repeats=True)
    assert np.all(st == L.S_OK)
    assert np.all(np.isfinite(lat)) and np.all(lat > 0)
    for i in range(len(scheds)):
        assert lat[i] == HR.median(rep[i])
    lat2, st2 = L.measure_candidates(op, scheds, 0.25, opts, xd, wd, yd)
    assert np.all(st2 == L.S_OK) and np.all(lat2 > 0)


def test_invalid_schedules_are_not_launched():
    op = W.config(1).ops[0]
    x, w = make_inputs(op, "uniform", config_id=1)
    xd, wd, yd = to_device(op, x, w)
    good = L.ct_sample(op, 0, 1, 0, 2)
    bad = L.make_schedule(W.FAM_IGEMM_BF16, [16, 1, 1, 1, 1, 32, 0, 1, 0])  # wrong dtype/layout
    note("measure with invalid schedule")
    lat, st = L.measure_candidates(op, [good[0], bad, good[1]], 1.0, L.make_opts(1, 3, 2, 4), xd, wd, yd)
    assert list(st) == [L.S_OK, L.S_INVALID, L.S_OK]
    assert np.isinf(lat[1])


def test_verification_flags_a_corrupted_reference():
    op = W.conv("v", 1, 16, 20, 24, 3, 1)
    x, w = make_inputs(op, "uniform", seed=5)
    ref, _ = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    good_ref = torch.from_numpy(ref.astype(np.float32)).cuda()
    bad = ref.astype(np.float32).copy()
    bad.reshape(-1)[123] += 0.5
    bad_ref = torch.from_numpy(bad).cuda()
    scheds = L.ct_sample(op, 3, 0, 0, 12)
    opts = L.make_opts(1, 3, 2, 5)
    note("verify with the true reference")
    _, st = L.measure_candidates_mask(op, scheds, None, opts, xd, wd, yd, y_ref=good_ref, tol=1e-4)
    assert np.all(st == L.S_OK)
    note("verify with a corrupted reference")
    _, st = L.measure_candidates_mask(op, scheds, None, opts, xd, wd, yd, y_ref=bad_ref, tol=1e-4)
    assert np.all(st == L.S_WRONG_ANSWER)


def test_empty_kernel_floor_and_copy_bandwidth():
    opts = L.make_opts(2, 5, 20, 1)
    for f in (0.25, 1.0):
        note("empty probe fraction %.2f" % f)
        us = L.ct_probe_empty(L.ct_cu_mask(f, 0), 1, opts)
        assert 0 < us < 100
    nbytes = 256 << 20
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    note("copy probe")
    g = L.ct_probe_copy(L.ct_cu_mask(1.0, 0), src, dst, nbytes, L.make_opts(1, 3, 2, 1))
    assert 500 < g < 10000
