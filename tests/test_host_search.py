"""Guided search proposals (section 2.1, stage 4): host-only checks of the
annealing explorer and its cost model on synthetic latency functions whose
optimum is known by brute force over the valid space."""
import numpy as np
import pytest

from paper_2008_03602_amd import _lib as L, workloads as W

OP = W.config(2).ops[1]  # ResNet-18 3x3 64->64 at 56x56: direct and fp32 MFMA families


def _key(s):
    return (s.family,) + tuple(s.knob)


def _additive(seed):
    """Latency = exp(sum of a random weight per (family, knob, value)): a
    function the cost model can represent exactly."""
    rng = np.random.default_rng(seed)
    tab = {}

    def f(s):
        v = 0.0
        for k in range(L.MAX_KNOBS):
            key = (s.family, k, s.knob[k])
            if key not in tab:
                tab[key] = rng.uniform(0.0, 1.0)
            v += tab[key]
        return float(np.exp(v))
    return f


@pytest.fixture(scope="module")
def space():
    return L.ct_valid_space(OP)


def _run(f, so, rounds, failing=()):
    meas, lat, st = [], [], []
    for r in range(rounds):
        p = L.ct_search_propose(OP, meas, np.array(lat, np.float32), np.array(st, np.int32), so, r)
        for s in p:
            meas.append(s)
            bad = _key(s) in failing
            lat.append(np.inf if bad else f(s))
            st.append(L.S_TIMEOUT if bad else L.S_OK)
    return meas, np.array(lat), np.array(st)


def test_first_round_is_uniform_distinct_and_valid(space):
    so = L.make_search_opts(seed=5, batch=32)
    p = L.ct_search_propose(OP, [], [], [], so, 0)
    assert len(p) == 32
    assert len({_key(s) for s in p}) == 32
    assert all(L.ct_validate(OP, s) == 0 for s in p)
    fams = {s.family for s in p}
    assert fams <= {1, 4}


def test_proposals_are_deterministic_and_new(space):
    f = _additive(1)
    so = L.make_search_opts(seed=7, batch=16)
    meas, lat, st = _run(f, so, 3)
    a = L.ct_search_propose(OP, meas, lat.astype(np.float32), st, so, 3)
    b = L.ct_search_propose(OP, meas, lat.astype(np.float32), st, so, 3)
    assert [_key(s) for s in a] == [_key(s) for s in b]
    seen = {_key(s) for s in meas}
    assert len(a) == 16 and len({_key(s) for s in a}) == 16
    assert not seen & {_key(s) for s in a}
    assert all(L.ct_validate(OP, s) == 0 for s in a)
    c = L.ct_search_propose(OP, meas, lat.astype(np.float32), st, L.make_search_opts(seed=8, batch=16), 3)
    assert [_key(s) for s in c] != [_key(s) for s in a]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_guided_search_finds_the_optimum_of_a_representable_cost(space, seed):
    # the cost model fits an additive log latency exactly, so annealing on it
    # must reach the brute-force optimum within 16 rounds of 16: 256
    # measurements, 0.2 % of this space (seeds 0-7 need 3 to 15 rounds)
    f = _additive(seed)
    best = min(f(s) for s in space)
    so = L.make_search_opts(seed=seed, batch=16)
    _, lat, _ = _run(f, so, 16)
    assert lat.min() == pytest.approx(best, rel=1e-6)
    # uniform sampling with the same budget does not reach it on this space
    rng = np.random.default_rng(seed)
    rand = min(f(space[i]) for i in rng.choice(len(space), size=256, replace=False))
    assert rand > best * (1 + 1e-6)


def test_guided_batches_beat_uniform_batches(space):
    # explore = 1 turns the search into uniform sampling; the default mix of
    # model picks and uniform draws must do better on the same budget
    for seed in (4, 5):
        f = _additive(seed)
        best = min(f(s) for s in space)
        _, lat_g, _ = _run(f, L.make_search_opts(seed=seed, batch=16), 6)
        _, lat_u, _ = _run(f, L.make_search_opts(seed=seed, batch=16, explore=1.0), 6)
        assert lat_g.min() < lat_u.min()
        assert lat_g.min() < 1.05 * best


def test_failed_measurements_are_not_proposed_again_and_do_not_train(space):
    f = _additive(2)
    so = L.make_search_opts(seed=3, batch=16)
    first = L.ct_search_propose(OP, [], [], [], so, 0)
    failing = {_key(s) for s in first[:8]}
    meas, lat, st = _run(f, so, 4, failing=failing)
    keys = [_key(s) for s in meas]
    assert len(keys) == len(set(keys))
    assert np.sum(st == L.S_TIMEOUT) == 8


def test_bad_arguments_are_refused():
    so = L.make_search_opts(batch=0)
    with pytest.raises(L.CtError):
        L.ct_search_propose(OP, [], [], [], so, 0)
    so = L.make_search_opts(explore=1.5)
    with pytest.raises(L.CtError):
        L.ct_search_propose(OP, [], [], [], so, 0)
    bad = L.make_schedule(1, [3] * 9)  # values outside the knob tables
    with pytest.raises(L.CtError):
        L.ct_search_propose(OP, [bad], [1.0], [0], L.make_search_opts(), 1)


def test_small_space_runs_out_cleanly():
    # a bf16 pointwise op with few valid schedules: repeated rounds end with
    # fewer proposals than the batch and never repeat one
    op = W.Op("tiny", 1, 8, 4, 4, 8, 1, 1, 1, 1, 0, 0, 1, 1, 1, W.DT_BF16, W.LAYOUT_NHWC)
    n_space = len(L.ct_valid_space(op))
    so = L.make_search_opts(seed=0, batch=256, budget=100000)
    meas = []
    for r in range(n_space // 256 + 3):
        p = L.ct_search_propose(op, meas, np.ones(len(meas), np.float32), np.zeros(len(meas), np.int32), so, r)
        if not p:
            break
        meas += p
    assert len(meas) == n_space
    assert len({_key(s) for s in meas}) == n_space
