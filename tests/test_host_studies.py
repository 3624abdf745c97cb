"""Host-side post-processing of the studies: model-level aggregates of the
cross-evaluation (the model tables of section 4.1) and layer multiplicities."""
import numpy as np
import pytest

from paper_2008_03602_amd import tuner as T, workloads as W


def test_multiplicities_count_every_convolution():
    # ResNet-18: stem + 16 3x3 + projections at the four stage entries = 21;
    # ResNet-50 bottlenecks without the stem: 16 x 3 + 4 projections = 52
    assert sum(W.multiplicity(o.name) for o in W.config(2).ops) == 21
    assert sum(W.multiplicity(o.name) for o in W.resnet50()) == 52
    assert W.multiplicity("no-such-layer") == 1


def test_model_aggregates_by_hand():
    fr = (0.25, 1.0)
    # rows: tuned at f, columns: run at g (microseconds)
    m = {"r18.1": [[10.0, 4.0], [12.0, 3.0]],   # multiplicity 1
         "r18.2": [[5.0, 2.0], [6.0, 2.5]]}      # multiplicity 4
    agg = T.model_aggregates(m, fr)
    total = [[10 + 4 * 5, 4 + 4 * 2], [12 + 4 * 6, 3 + 4 * 2.5]]  # [[30, 12], [36, 13]]
    best = [10 + 4 * 5, 3 + 4 * 2]                                # per column, layer by layer: [30, 11]
    assert np.allclose(agg["total_us"], total)
    assert np.allclose(agg["best_us"], best)
    ratio = np.array(total) / np.array(best)[None, :]
    assert np.allclose(agg["ratio_to_best"], ratio)
    assert np.allclose(agg["mean_ratio_per_tuning_share"], ratio.mean(axis=1))
    # tuned at 25%: (1 + 12/11)/2 = 1.045; at 100%: (1.2 + 13/11)/2 = 1.191
    assert agg["sweet_spot"] == 0.25


def test_model_aggregates_diagonal_matrix_picks_nothing_worse_than_best():
    rng = np.random.default_rng(3)
    fr = (0.125, 0.25, 0.5, 1.0)
    m = {}
    for i in range(5):
        base = rng.uniform(5, 50, size=4)
        M = base[None, :] * rng.uniform(1.0, 1.5, size=(4, 4))
        np.fill_diagonal(M, base)      # each share's own winner is the fastest at that share
        m["r18.%d" % (i + 1)] = M.tolist()
    agg = T.model_aggregates(m, fr)
    ratio = np.array(agg["ratio_to_best"])
    assert np.allclose(np.diag(ratio), 1.0)
    assert np.all(ratio >= 1.0 - 1e-12)
    assert agg["sweet_spot"] in fr


def test_regret_is_one_on_the_diagonal_of_a_consistent_matrix():
    M = [[1.0, 3.0], [2.0, 2.0]]
    r = T.cross_eval_regret({"a": M}, (0.5, 1.0))
    assert np.allclose(r, [[1.0, 1.5], [2.0, 1.0]])
