"""GPU tests of the boundary calls added around measurement: registered
references (the runner's correctness check), the stream pool, one client over
several CU slots, and the timeout watchdog on a real stream."""
import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, tuner as T, workloads as W
from gpu_util import device_ready, make_inputs, note, reference, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def test_registered_reference_sets_wrong_answer():
    op = W.conv("refop", 1, 16, 20, 24, 3, 1)
    x, w = make_inputs(op, "uniform", seed=5)
    ref, _ = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    scheds = L.ct_sample(op, 3, 0, 0, 10)
    opts = L.make_opts(1, 3, 2, 4)
    try:
        L.ct_set_reference(op, ref)
        note("measure with the registered true reference")
        _, st = L.measure_candidates(op, scheds, 0.25, opts, xd, wd, yd)
        assert np.all(st == L.S_OK)
        bad = ref.copy()
        bad.reshape(-1)[77] += 0.25
        L.ct_set_reference(op, bad)
        note("measure with a registered corrupted reference")
        _, st = L.measure_candidates(op, scheds, 0.25, opts, xd, wd, yd)
        assert np.all(st == L.S_WRONG_ANSWER)
        # an explicit reference takes precedence over the registered one
        _, st = L.measure_candidates_mask(op, scheds, L.ct_cu_mask(0.25, 0), opts, xd, wd, yd,
                                          y_ref=torch.from_numpy(ref.astype(np.float32)).cuda(), tol=1e-4)
        assert np.all(st == L.S_OK)
    finally:
        L.ct_set_reference(op, None)
    _, st = L.measure_candidates(op, scheds, 0.25, opts, xd, wd, yd)
    assert np.all(st == L.S_OK)


def test_registered_reference_covers_bf16_tolerance():
    op = W.conv("refbf", 2, 40, 9, 48, 1, 1, 0, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC)
    x, w = make_inputs(op, "uniform", seed=6)
    ref, _ = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    scheds = L.ct_sample(op, 4, 0, 0, 8)
    try:
        L.ct_set_reference(op, ref)
        note("bf16 measure with registered reference")
        _, st = L.measure_candidates(op, scheds, 0.5, L.make_opts(1, 2, 2, 4), xd, wd, yd)
        assert np.all(st == L.S_OK)
    finally:
        L.ct_set_reference(op, None)


def test_streams_are_reused_across_tuning_calls():
    cfg = W.config(2)
    cfg.n_candidates = 8
    cfg.top_t = 2
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops[:4])]
    cands = T.sample_all(layers, cfg)
    note("stream pool: 3 rounds of 4 clients at 25%")
    T.tune_model_at_fraction(layers, cands, cfg, 0.25)
    n0 = L.ct_stream_count()
    for _ in range(3):
        T.tune_model_at_fraction(layers, cands, cfg, 0.25)
        T.cross_eval(layers[0], [cands[0][0], cands[0][1]], [L.ct_cu_mask(0.25, 0)], cfg.stage2)
    assert L.ct_stream_count() == n0


@pytest.mark.parametrize("k", [1, 2, 4])
def test_one_client_over_k_slots_matches_the_oracle(k):
    cfg = W.config(2)
    cfg.n_candidates = 24
    cfg.top_t = 4
    ld = T.make_layer(cfg.ops[1], cfg, 1)
    c = L.ct_sample(ld.op, cfg.seed, cfg.config_id, 1, cfg.n_candidates)
    x, w = make_inputs(ld.op, cfg.dist, seed=cfg.seed, config_id=cfg.config_id, layer_id=1)
    ref, _ = reference(ld.op, x, w, threads=16)
    yref = torch.from_numpy(ref.astype(np.float32)).cuda()
    ys = [ld.y] + [torch.empty_like(ld.y) for _ in range(k - 1)]
    note("ct_tune_split k=%d on r18.2" % k)
    r = T.tune_split(ld, c, cfg, 0.25, k, ys, y_ref=yref)
    res = r["result"]
    assert r["status_counts"] == {"ok": len(c)}
    assert np.all(np.isfinite(res.lat1)) and res.winner_pos >= 0
    # the winner is among the merged stage-1 top_t and has the lowest position in the tie band
    assert res.winner_pos in set(res.top_pos.tolist())
    lim = float(np.min(res.lat2)) * (1 + cfg.eps)
    tied = [int(p) for p, l in zip(res.top_pos, res.lat2) if l <= lim]
    assert res.winner_pos == min(tied)
    assert r["screen_s"] > 0 and r["total_s"] >= r["screen_s"]


def test_timeout_fires_on_a_slow_candidate_and_the_stream_stays_usable():
    # 8 CUs (one per XCD; a queue needs CUs on every XCD): one 64->64 3x3 56x56
    # run takes about 0.2 ms or more (231 MFLOP at 1/32 of the fp32 peak is
    # 47 us, and the best schedules reach a fifth of the peak), so 1000
    # back-to-back runs exceed a 0.01 ms-per-run limit by far more than the
    # 50 ms slack
    cfg = W.config(2)
    ld = T.make_layer(cfg.ops[1], cfg, 1)
    s = next(s for s in L.ct_sample(ld.op, 0, 2, 1, 16) if s.family == W.FAM_IGEMM_F32)
    mask = L.ct_cu_mask(8.0 / 256, 0)
    assert sum(bin(int(v)).count("1") for v in mask) == 8
    note("timeout: F4 schedule on 8 CUs with a 0.01 ms limit")
    lat, st = L.measure_candidates_mask(ld.op, [s], mask, L.make_opts(1, 2, 1000, 1, timeout_ms=0.01),
                                        ld.x, ld.w, ld.y)
    assert st[0] == L.S_TIMEOUT
    note("same mask, normal limit")
    lat, st = L.measure_candidates_mask(ld.op, [s], mask, L.make_opts(1, 2, 4, 1, timeout_ms=1000.0),
                                        ld.x, ld.w, ld.y)
    assert st[0] == L.S_OK and lat[0] > 40.0
