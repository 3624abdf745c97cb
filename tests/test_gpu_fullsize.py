"""Full-size parity of the ResNet-50 b1 and MobileNet-v2 b16 workloads on the
GPU: every layer at its real shape, sampled schedules from the workload's own
seeded candidate list, on the 25 % slot-0 stream the tuning clients use.

Per layer: 8 sampled schedules checked on the device against the fp64 oracle
(infinity-norm relative error 1e-4 for fp32, 2e-2 for bf16), two of them
compared element by element on the host against the oracle and the fp32
summation bound, and one schedule per applicable kernel family run on integer
inputs, whose output must equal the oracle's bit for bit."""
import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, workloads as W
from gpu_util import check_close, device_ready, make_inputs, note, reference, sched_str, to_device

pytestmark = pytest.mark.gpu

CFG4 = W.config(4)
CFG5 = W.config(5)
CASES = [(4, i) for i in range(len(CFG4.ops))] + [(5, i) for i in range(len(CFG5.ops))]


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _case_id(c):
    cfg = CFG4 if c[0] == 4 else CFG5
    return cfg.ops[c[1]].name


@pytest.mark.parametrize("case", CASES, ids=_case_id)
def test_full_size_layer_matches_oracle(case):
    cid, layer = case
    cfg = CFG4 if cid == 4 else CFG5
    op = cfg.ops[layer]
    bf16 = op.dtype == W.DT_BF16
    tol = 2e-2 if bf16 else 1e-4
    x, w = make_inputs(op, cfg.dist, seed=cfg.seed, config_id=cfg.config_id, layer_id=layer)
    ref, a = reference(op, x, w, threads=16)
    xd, wd, yd = to_device(op, x, w)
    yref = torch.from_numpy(ref.astype(np.float32)).to("cuda:0")
    sample = L.ct_sample(op, cfg.seed, cfg.config_id, layer, cfg.n_candidates)
    scheds = sample[:8]
    note("full-size %s: %d schedules verified on the 25%% slot" % (op.name, len(scheds)))
    lat, st = L.measure_candidates_mask(op, scheds, L.ct_cu_mask(0.25, 0), L.make_opts(1, 1, 1, 4), xd, wd, yd,
                                        y_ref=yref, tol=tol)
    bad = [sched_str(s) for s, v in zip(scheds, st) if v != L.S_OK]
    assert not bad, "%s: %s" % (op.name, bad)
    for s in scheds[:2]:
        note("full-size %s element-wise %s" % (op.name, sched_str(s)))
        yd.fill_(float("nan"))
        L.conv2d_run(op, s, xd, wd, yd, L.ct_cu_mask(0.25, 0))
        check_close(op, yd.cpu().numpy(), ref, a, "%s %s" % (op.name, sched_str(s)), split=8)

    # integer inputs: fp32 x, w in {-2..2}; bf16 x, w in {-8..8} (exact in bf16);
    # every partial sum is an integer below 2^24, so any order is exact
    xi, wi = make_inputs(op, "int", seed=cfg.seed + 7, layer_id=layer, int_range=8 if bf16 else 2)
    refi, _ = reference(op, xi, wi, threads=16)
    xid, wid, yid = to_device(op, xi, wi)
    fams = sorted({int(s.family) for s in sample})
    for fam in fams:
        s = next(s for s in sample if s.family == fam)
        note("full-size %s integer %s" % (op.name, sched_str(s)))
        yid.fill_(float("nan"))
        L.conv2d_run(op, s, xid, wid, yid, L.ct_cu_mask(0.25, 0))
        assert np.array_equal(yid.cpu().numpy().astype(np.float64), refi), \
            "%s %s: not bit-exact on integer inputs" % (op.name, sched_str(s))
