"""GPU tests of the tuning path: determinism, concurrent clients, CU-share
scaling, the cross-evaluation diagonal, and full-size layers verified on the
masked streams the tuner times them on.
"""
import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, tuner as T, workloads as W
from gpu_util import check_close, device_ready, make_inputs, note, reference, sched_str, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _small_cfg(n_candidates=24, top_t=4):
    cfg = W.config(2)
    cfg.n_candidates = n_candidates
    cfg.top_t = top_t
    return cfg


def test_candidate_lists_identical_across_runs_and_fractions():
    cfg = _small_cfg()
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops[:3])]
    a = {k: [L.schedule_tuple(s) for s in v] for k, v in T.sample_all(layers, cfg).items()}
    b = {k: [L.schedule_tuple(s) for s in v] for k, v in T.sample_all(layers, cfg).items()}
    assert a == b
    note("tune 3 layers at 25% and 100%")
    cands = T.sample_all(layers, cfg)
    r25 = T.tune_model_at_fraction(layers, cands, cfg, 0.25)
    r100 = T.tune_model_at_fraction(layers, cands, cfg, 1.0)
    for x in r25 + r100:
        assert [L.schedule_tuple(s) for s in x.candidates] == a[x.layer_id]


def test_winner_repeats_or_ties_for_a_fixed_seed():
    # the winner is the lowest stage-2 latency, with anything within eps of it
    # tied and resolved by sample position; a rerun must pick the same
    # schedule or one whose latencies sit in the tie band of both runs
    cfg = _small_cfg(n_candidates=32, top_t=8)
    op = W.config(1).ops[0]
    ld = T.make_layer(op, cfg, 0)
    cands = {0: L.ct_sample(op, cfg.seed, 1, 0, cfg.n_candidates)}
    runs = []
    for r in range(2):
        note("tune config1 layer run %d" % r)
        runs.append(T.tune_clients([[ld]], [L.ct_cu_mask(1.0, 0)], cands, cfg, 1.0)[0])
    w0, w1 = runs[0].winner_pos, runs[1].winner_pos
    assert w0 >= 0 and w1 >= 0
    if w0 != w1:
        m = L.make_opts(2, 21, 10, 2, interleave=1)
        lat, st = L.measure_candidates_mask(op, [cands[0][w0], cands[0][w1]], L.ct_cu_mask(1.0, 0), m,
                                            ld.x, ld.w, ld.y)
        assert np.all(st == L.S_OK)
        gap = abs(lat[0] - lat[1]) / min(lat)
        print("winner flip %d -> %d, re-measured gap %.2f%%" % (w0, w1, 100 * gap))
        assert gap <= 0.03, "winners differ by %.1f%%, beyond the tie band" % (100 * gap)


def test_four_clients_run_concurrently_match_the_oracle_and_double_one():
    # the multi-client workload: ResNet-50 b1's 22 bottleneck layers, four
    # clients on disjoint 64-CU slots against one client on all 256 CUs, every
    # screened candidate's output checked on the device against the oracle
    cfg = W.config(4)
    cfg.n_candidates = 32
    cfg.top_t = 4
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops)]
    refs = {}
    for ld in layers:
        x, w = make_inputs(ld.op, cfg.dist, seed=cfg.seed, config_id=cfg.config_id, layer_id=ld.layer_id)
        ref, _ = reference(ld.op, x, w, threads=16)
        refs[ld.layer_id] = torch.from_numpy(ref.astype(np.float32)).to("cuda:0")
    cands = T.sample_all(layers, cfg)
    note("4 clients x 22 ResNet-50 layers at 25%, verified")
    four = T.tune_model_at_fraction(layers, cands, cfg, 0.25, verify_refs=refs)
    for r in four:
        assert r.winner_pos >= 0
        assert np.all(r.status1 == L.S_OK), (r.op.name, r.summary()["status_counts"])
    spans = {}
    for r in four:
        s, e = spans.get(r.client, (np.inf, -np.inf))
        spans[r.client] = (min(s, r.t_start), max(e, r.t_end))
    assert len(spans) == 4
    assert max(s for s, _ in spans.values()) < min(e for _, e in spans.values()), "clients did not overlap"
    note("1 client x 22 ResNet-50 layers at 100%, verified")
    one = T.tune_model_at_fraction(layers, cands, cfg, 1.0, verify_refs=refs)
    assert all(np.all(r.status1 == L.S_OK) for r in one)
    # throughput without the verification re-runs, on 128 candidates per layer
    # (a quarter of the workload's 512: the re-measure of the top 4 weighs about
    # as much against the screen as the full workload's top 8 against 512)
    cfg.n_candidates = 128
    cands = T.sample_all(layers, cfg)
    note("4 clients at 25% and 1 client at 100%, timed, 128 candidates per layer")
    four = T.tune_model_at_fraction(layers, cands, cfg, 0.25)
    one = T.tune_model_at_fraction(layers, cands, cfg, 1.0)
    f4, f1 = T.fraction_report(four), T.fraction_report(one)
    ratio = f4["candidates_per_s"] / f1["candidates_per_s"]
    print("candidates/s: 4 clients %.1f (per client %s), 1 client %.1f, ratio %.2f" % (
        f4["candidates_per_s"], np.round(f4["per_client_candidates_per_s"], 1).tolist(), f1["candidates_per_s"],
        ratio))
    # the full 512-candidate workload reaches 2x (a tuning run of the whole
    # configuration); this quarter-size sample keeps a margin for run-to-run spread
    assert ratio >= 1.9


def test_shared_queue_runs_every_layer_once_and_matches_round_robin_lists():
    cfg = _small_cfg(n_candidates=12, top_t=2)
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops[:6])]
    cands = T.sample_all(layers, cfg)
    note("shared queue: 3 clients x 6 layers at 25%")
    masks = [L.ct_cu_mask(0.25, j) for j in range(3)]
    res = T.tune_shared(T.largest_first(layers), masks, cands, cfg, 0.25)
    assert sorted(r.layer_id for r in res) == list(range(6))
    assert all(0 <= r.client < 3 and r.winner_pos >= 0 for r in res)
    assert all(np.all(r.status1 == L.S_OK) for r in res)
    # each client's jobs run one after another
    for c in range(3):
        spans = sorted((r.t_start, r.t_end) for r in res if r.client == c)
        assert all(a[1] <= b[0] + 1e-6 for a, b in zip(spans, spans[1:]))
    for r in res:
        assert [L.schedule_tuple(s) for s in r.candidates] == [L.schedule_tuple(s) for s in cands[r.layer_id]]


def test_compute_bound_latency_scales_with_cu_share():
    op = W.config(1).ops[0]
    cfg = _small_cfg()
    ld = T.make_layer(op, cfg, 0)
    # a direct schedule with many small blocks: the grid is much larger than
    # the device, so the time tracks the number of CUs
    s = L.make_schedule(1, [1, 8, 16, 2, 1, 1, 16, 1, 1])
    assert L.ct_validate(op, s) == 0, L.ct_last_error()
    assert L.ct_launch_shape(op, s)["blocks"] >= 4 * L.ct_num_cus()
    o = L.make_opts(2, 5, 10, 1)
    lat = {}
    for f in (0.25, 0.5, 1.0):
        note("scaling probe at %.2f" % f)
        lt, st = L.measure_candidates_mask(op, [s], L.ct_cu_mask(f, 0), o, ld.x, ld.w, ld.y)
        assert st[0] == L.S_OK
        lat[f] = float(lt[0])
    print("latency by share:", lat)
    assert lat[0.25] > 2.5 * lat[1.0]
    assert lat[0.5] > 1.4 * lat[1.0]


def test_cross_eval_diagonal_is_best_in_its_column():
    # best_f was chosen on share f from the same list as best_g, so on share f
    # it is not slower than best_g beyond measurement noise
    cfg = _small_cfg(n_candidates=24, top_t=6)
    op = W.config(2).ops[1]
    ld = T.make_layer(op, cfg, 1)
    cands = {1: L.ct_sample(op, cfg.seed, cfg.config_id, 1, cfg.n_candidates)}
    fr = (0.25, 1.0)
    winners = []
    for f in fr:
        note("tune r18.2 at %.2f" % f)
        winners.append(T.tune_clients([[ld]], [L.ct_cu_mask(f, 0)], cands, cfg, f)[0].winner)
    masks = [L.ct_cu_mask(f, 0) for f in fr]
    M = T.cross_eval(ld, winners, masks, cfg.stage2)
    print("cross-eval (us):", M.tolist())
    for j in range(len(fr)):
        assert M[j][j] <= 1.03 * M[:, j].min(), "share %.2f: own winner %.2f us vs best %.2f us" % (
            fr[j], M[j][j], M[:, j].min())


@pytest.mark.parametrize("layer", range(12))
def test_full_size_resnet18_layers_verify_on_masked_streams(layer):
    # the first 12 candidates of the benchmark's 256-candidate sample of each
    # layer (both kernel families), at full size, on the 25% slot-0 stream the
    # tuner uses, checked on the device against the oracle; the last two
    # outputs are then compared element by element
    cfg = W.config(2)
    op = cfg.ops[layer]
    x, w = make_inputs(op, cfg.dist, seed=cfg.seed, config_id=cfg.config_id, layer_id=layer)
    ref, a = reference(op, x, w, threads=16)
    xd, wd, yd = to_device(op, x, w)
    yref = torch.from_numpy(ref.astype(np.float32)).to("cuda:0")
    scheds = L.ct_sample(op, cfg.seed, cfg.config_id, layer, 12)
    o = L.make_opts(1, 1, 1, 4)
    note("verify %s, %d candidates at 25%%" % (op.name, len(scheds)))
    lat, st = L.measure_candidates_mask(op, scheds, L.ct_cu_mask(0.25, 0), o, xd, wd, yd, y_ref=yref,
                                        tol=1e-4)
    bad = [sched_str(s) for s, v in zip(scheds, st) if v != L.S_OK]
    assert not bad, "%s: %s" % (op.name, bad)
    for s in scheds[-2:]:
        yd.fill_(float("nan"))
        L.conv2d_run(op, s, xd, wd, yd)
        check_close(op, yd.cpu().numpy(), ref, a, "%s %s" % (op.name, sched_str(s)), split=8)


def test_empty_candidate_list_and_a_layer_that_fails_verification():
    # degenerate cases of a tuning run: no candidates to measure; a layer whose
    # every candidate fails verification (its reference is wrong on purpose)
    # ends with no winner while the other layer of the run tunes normally
    cfg = W.config(2)
    cfg.n_candidates = 8
    cfg.top_t = 4
    layers = [T.make_layer(op, cfg, i) for i, op in enumerate(cfg.ops[:2])]
    note("measure an empty candidate list")
    lat, st = L.measure_candidates_mask(layers[0].op, [], L.ct_cu_mask(0.25, 0), L.make_opts(1, 2, 2),
                                        layers[0].x, layers[0].w, layers[0].y)
    assert lat.size == 0 and st.size == 0
    refs = {}
    for ld in layers:
        x, w = make_inputs(ld.op, cfg.dist, seed=cfg.seed, config_id=cfg.config_id, layer_id=ld.layer_id)
        ref, _ = reference(ld.op, x, w, threads=16)
        if ld.layer_id == 1:
            ref = ref + 1.0  # every output off by one: no schedule can match
        refs[ld.layer_id] = torch.from_numpy(ref.astype(np.float32)).to("cuda:0")
    cands = T.sample_all(layers, cfg)
    note("two layers, the second with a wrong reference, two clients at 25%")
    res = T.tune_model_at_fraction(layers, cands, cfg, 0.25, verify_refs=refs)
    good, bad = res[0], res[1]
    assert good.winner_pos >= 0 and np.all(good.status1 == L.S_OK)
    assert bad.winner_pos == -1 and np.all(bad.status1 == L.S_WRONG_ANSWER)
    assert bad.winner_lat_us == float("inf")
