"""GPU checks of the studies: one layer's candidates spread over several CU
slots (TSI scaling), latency isolation of a masked slot, and the guided
search against the random-sample tuner."""
import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, studies as S, tuner as T, workloads as W
from gpu_util import device_ready, make_inputs, note, reference


def _ref_of(ld, cfg):
    """The oracle's output of a layer's seeded inputs, as an fp32 device tensor."""
    x, w = make_inputs(ld.op, cfg.dist, seed=cfg.seed, config_id=cfg.config_id, layer_id=ld.layer_id)
    ref, _ = reference(ld.op, x, w, threads=16)
    return torch.from_numpy(ref.astype(np.float32)).to("cuda:0")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _cfg(n_candidates, top_t=4):
    cfg = W.config(2)
    cfg.n_candidates = n_candidates
    cfg.top_t = top_t
    return cfg


def test_split_screening_is_faster_and_keeps_the_winner():
    # the workload's own re-measure depth (top 8)
    cfg = _cfg(48, top_t=8)
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops[:2])]
    cands = T.sample_all(layers, cfg)
    refs = {ld.layer_id: _ref_of(ld, cfg) for ld in layers}
    note("tsi: 2 layers x k in (1, 4), outputs checked against the oracle")
    rep = S.tsi_scaling(layers, cands, cfg, fraction=0.25, ks=(1, 4), verify_refs=refs)
    for row in rep["layers"]:
        for r in row["runs"]:
            # every candidate of every slot ran, matched the oracle and was timed
            assert r["screened_ok"] == row["candidates"], row
            assert r["status_counts"] == {"ok": row["candidates"]}, row
            assert r["winner_pos"] >= 0
        # k slots screen side by side, and busy neighbours inflate a slot's
        # latencies unevenly (by up to 1.16x for the same kernels in the
        # isolation study), so the k-slot screen may rank the single-slot
        # winner out of its top 8; the winner it then picks, re-measured
        # alone, stays within that inflation of the single-slot winner
        flip = row["runs"][1]
        if flip["winner_pos"] != row["runs"][0]["winner_pos"]:
            assert flip["flip_gap"] <= 0.16, row
    print("tsi speedup:", rep["speedup"])
    assert rep["speedup"]["4"] > 1.5


def test_masked_slot_latency_holds_with_compute_neighbours():
    cfg = _cfg(32)
    op = cfg.ops[1]
    ld = T.make_layer(op, cfg, 1)
    cands = L.ct_sample(op, cfg.seed, cfg.config_id, 1, 32)
    note("isolation: r18.2, 4 schedules (%d library streams)" % L.ct_stream_count())
    with S.Slots(4) as slots:
        ys = [ld.y] + [ld.y.new_empty(ld.y.shape) for _ in range(3)]
        n = 64 << 18
        bufs = [(ld.y.new_ones(n), ld.y.new_empty(n)) for _ in range(3)]
        lat, st = L.measure_candidates_mask(op, cands, L.ct_cu_mask(0.25, 0), L.opts_from_protocol(cfg.stage1),
                                            ld.x, ld.w, ld.y)
        top = L.ct_top_t(lat, st, 4)
        r = S.isolation(ld, [cands[i] for i in top], cfg, slots, bufs, ys, y_ref=_ref_of(ld, cfg))
    print("inflation:", {k: np.round(v, 3).tolist() for k, v in r["inflation"].items()})
    # the timed slot's outputs match the oracle whatever its neighbours run
    for k, st in r["status"].items():
        assert st == [L.S_OK] * len(top), (k, st)
    for k, v in r["latency_us"].items():
        assert np.all(np.isfinite(v)), k
    # four disjoint 64-CU slots running conv kernels: the masked latency moves by
    # a few percent (HBM and L2 are shared, the CUs are not)
    assert np.median(r["inflation"]["neighbours_same_kernels"]) < 1.3
    assert min(min(v) for v in r["inflation"].values()) > 0.85


def test_guided_search_reaches_the_random_winner_on_a_layer():
    # budget 256 (the search study's): the fp32 MFMA grid holds about 25k
    # schedules of this layer, and the cost model needs a few batches of them
    # before its proposals beat random picks; its proposals follow measured,
    # noisy latencies, so a budget near the edge fails now and then (160 came
    # 5.4 % off once)
    cfg = _cfg(256, top_t=4)
    layers = [T.make_layer(cfg.ops[1], cfg, 1)]
    cands = T.sample_all(layers, cfg)
    note("guided search vs random, r18.2 at 25%, budget 256")
    rep = S.search_study(layers, cands, cfg, fraction=0.25, within=0.05, patience=32)
    row = rep["layers"][0]
    print(row)
    assert row["guided_to_within"] > 0, "guided search never came within 5% of the random winner"
    assert row["guided_winner_us"] <= 1.10 * row["random_winner_us"]
    assert 0 < row["early_stop_measured"] <= row["budget"]


def test_search_entry_point_measures_distinct_valid_candidates():
    cfg = _cfg(32)
    op = cfg.ops[2]
    ld = T.make_layer(op, cfg, 2)
    so = L.make_search_opts(seed=11, batch=8, budget=40, patience=0)
    note("ct_search r18.3 budget 40")
    meas, lat, st, res = L.ct_search(op, so, L.ct_cu_mask(0.5, 0), L.opts_from_protocol(cfg.stage1),
                                     L.opts_from_protocol(cfg.stage2, batch=4, interleave=1), 4, cfg.eps,
                                     ld.x, ld.w, ld.y)
    assert res["n_measured"] == 40 and res["rounds"] == 5 and not res["stopped_early"]
    keys = {(s.family,) + tuple(s.knob) for s in meas}
    assert len(keys) == 40
    assert all(L.ct_validate(op, s) == 0 for s in meas)
    assert np.all(st == L.S_OK)
    assert 0 <= res["winner"] < 40 and np.isfinite(res["winner_lat_us"])
    # the winner is among the stage-1 top 4
    assert res["winner"] in set(L.ct_top_t(lat, st, 4).tolist())
