"""bench.py's host side (no GPU): the one-GPU refusal, the launch count that
scales the CPU baseline, and the CPU baseline's fields on a tiny budget."""
import os
import subprocess
import sys

import pytest

from paper_2008_03602_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_launches_per_candidate_by_hand():
    # one step, per layer: 3 shares x (32 x (2 + 5 x 10) screen + 8 x (2 + 21 x 10)
    # re-measure) + 9 x (2 + 21 x 10) cross-evaluation = 3 x (1664 + 1696) + 1908
    # = 11988 launches for 3 x 32 = 96 screened candidates: 124.875 each
    cfg = W.config(2)
    assert bench.launches_per_candidate(cfg, 12, 3, 32) == pytest.approx(11988 / 96, rel=0, abs=1e-12)
    assert bench.launches_per_candidate(cfg, 12, 3, 32) == pytest.approx(124.875, abs=1e-12)


def test_cpu_baseline_reports_its_sample_and_both_thread_counts():
    cfg = W.config(2)
    cb = bench.cpu_baseline(cfg, 124.875, budget_s=0.05, single_budget_s=0.05)
    assert cb["kind"] == "oracle" and cb["unit"] == "candidates/s"
    assert cb["cores"] == len(os.sched_getaffinity(0))
    assert cb["value"] == pytest.approx(cb["oracle_convs_per_s"] / 124.875)
    st = cb["single_thread"]
    assert st["cores"] == 1 and st["convolutions"] >= 1
    assert st["value"] == pytest.approx(st["oracle_convs_per_s"] / 124.875)
    assert "fp64 oracle convolutions" in cb["sample"] and "124.9" in cb["sample"]
