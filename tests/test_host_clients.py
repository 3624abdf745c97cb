"""Host logic of the tuning clients, on the CPU: the timeout watchdog, the
shared job queue, a failing client, per-client logs and resume.

The library's test entry points drive its own client threads, queue, logs and
selection with a stand-in for the device (ct_test_run_clients) and run the
watchdog on a simulated stream (ct_test_watchdog); nothing here computes a
convolution."""
import ctypes
import json
import os

import numpy as np
import pytest

from paper_2008_03602_amd import _lib as L
from paper_2008_03602_amd import tuner as T
from paper_2008_03602_amd import workloads as W


# ---------------------------------------------------------------- watchdog
def test_watchdog_all_in_time():
    ex, dr = L.ct_test_watchdog([2, 10, 10, 10], [0.001, 0.005, 0.009, 0.020], 0.002, 0.0, 1.0)
    assert (ex, dr) == (-1, True)


def test_watchdog_slow_event_then_drains():
    # event 2 is due 10 runs x 1 ms after event 1 completed (at 5 ms): 15 ms;
    # it completes at 40 ms, so its deadline passes; the stream then drains
    ex, dr = L.ct_test_watchdog([2, 10, 10, 10], [0.001, 0.005, 0.040, 0.041], 0.001, 0.0, 1.0)
    assert (ex, dr) == (2, True)


def test_watchdog_slack_absorbs_lateness():
    ex, dr = L.ct_test_watchdog([2, 10, 10, 10], [0.001, 0.005, 0.040, 0.041], 0.001, 0.05, 1.0)
    assert (ex, dr) == (-1, True)


def test_watchdog_never_drains():
    ex, dr = L.ct_test_watchdog([1, 10, 10], [0.0, -1.0, -1.0], 0.001, 0.0, 0.5)
    assert (ex, dr) == (1, False)


def test_watchdog_deadline_runs_from_previous_completion():
    # each event on its own is within budget (10 runs x 1 ms after the one before)
    done = [0.009 * (k + 1) for k in range(20)]
    ex, dr = L.ct_test_watchdog([10] * 20, done, 0.001, 0.0, 1.0)
    assert (ex, dr) == (-1, True)


def test_watchdog_rejects_bad_arguments():
    with pytest.raises(L.CtError):
        L.ct_test_watchdog([1], [0.0], 0.0, 0.0, 1.0)


# ---------------------------------------------------------------- clients
OP = W.conv("tiny", 1, 8, 8, 8, 3, 1)


def fake_lat(layer_id, i):
    """The stand-in latency the library documents for candidate i of a layer."""
    v = ((layer_id * 7919 + i) * 2654435761 % (1 << 64)) % 1000
    return np.float32(1.0) + np.float32(v) / np.float32(100.0)


def make_jobs(n_jobs, n_cands, keep, recorded=None, top_t=4):
    cands = L.ct_sample(OP, 0, 1, 0, n_cands)
    assert len(cands) == n_cands
    jobs = (L.ct_tune_job * n_jobs)()
    metas = []
    for i in range(n_jobs):
        metas.append(T.fill_job(jobs[i], OP, 100 + i, 1, 1, 1, cands, top_t, keep,
                                recorded=(recorded or {}).get(100 + i)))
    return jobs, metas, cands


def make_clients(k, logs=None, keep=None):
    return T._clients([np.zeros(L.MASK_WORDS, np.uint32)] * k, False, logs, keep)


def hooks(delay_us=0, throw_client=-1, throw_after_jobs=0, stop_after=-1):
    return L.ct_test_hooks(delay_us, throw_client, throw_after_jobs, stop_after)


def test_shared_queue_runs_every_job_once_and_selects_by_the_tie_rule():
    keep = T._Keep()
    jobs, metas, cands = make_jobs(7, 24, keep)
    clients = make_clients(3)
    owner = L.ct_test_run_clients(clients, jobs, hooks(delay_us=200))
    assert sorted(set(owner.tolist())) <= [0, 1, 2] and (owner >= 0).all()
    assert sum(c.n_measured for c in clients) == 7 * 24
    for i in range(7):
        lid = 100 + i
        lat1 = metas[i][1][:24]
        want = np.array([fake_lat(lid, p) for p in range(24)], np.float32)
        assert np.array_equal(lat1, want)
        # winner: the fastest by stage-1 order (the stand-in re-measure repeats it), lowest position on ties
        exp = min(range(24), key=lambda p: (want[p], p))
        assert jobs[i].winner_pos == exp and jobs[i].rc == 0
    for c in clients:
        assert c.rc == 0
        if c.n_measured:
            assert c.cands_per_s == pytest.approx(c.n_measured / (c.t_end_s - c.t_start_s))
    agg = L.ct_throughput(clients)
    span = max(c.t_end_s for c in clients) - min(c.t_start_s for c in clients)
    assert agg == pytest.approx(7 * 24 / span)


def test_raising_client_is_recorded_and_the_others_finish():
    keep = T._Keep()
    jobs, metas, _ = make_jobs(9, 8, keep)
    clients = make_clients(3)
    with pytest.raises(L.CtError) as e:
        L.ct_test_run_clients(clients, jobs, hooks(delay_us=500, throw_client=1, throw_after_jobs=1))
    assert e.value.code == L.CT_E_CLIENT
    assert "test hook raised" in str(e.value)
    assert clients[1].rc == L.CT_E_CLIENT and clients[0].rc == 0 and clients[2].rc == 0
    rcs = [jobs[i].rc for i in range(9)]
    assert rcs.count(L.CT_E_CLIENT) == 1          # the job the raising client had taken
    assert rcs.count(0) == 8                      # every other job ran to the end
    assert all(jobs[i].winner_pos >= 0 for i in range(9) if jobs[i].rc == 0)


def _read(path):
    with open(path) as fh:
        return [json.loads(l) for l in fh]


def test_logs_hold_every_candidate_and_job(tmp_path):
    keep = T._Keep()
    jobs, metas, cands = make_jobs(4, 10, keep)
    logs = [str(tmp_path / ("c%d.jsonl" % j)) for j in range(2)]
    clients = make_clients(2, logs, keep)
    owner = L.ct_test_run_clients(clients, jobs, hooks())
    recs = [r for p in logs if os.path.exists(p) for r in _read(p)]
    cand = [r for r in recs if r["kind"] == "cand"]
    job = [r for r in recs if r["kind"] == "job"]
    assert len(cand) == 40 and len(job) == 4
    for r in cand:
        s = cands[r["pos"]]
        assert r["family"] == s.family and r["knobs"] == list(s.knob[:len(r["knobs"])])
        assert np.float32(r["lat_us"]) == fake_lat(r["layer"], r["pos"]) and r["status"] == 0
    for r in job:
        i = r["layer"] - 100
        assert r["winner_pos"] == jobs[i].winner_pos
        # the job's records are in the log of the client that ran it
        assert any(rr["kind"] == "job" and rr["layer"] == r["layer"] for rr in _read(logs[owner[i]]))
    merged = T.read_logs(logs)
    assert merged["duplicates"] == 0 and set(merged["jobs"]) == {100, 101, 102, 103}


def test_stop_after_k_records_then_resume_measures_the_rest_once(tmp_path):
    n_jobs, n = 5, 12
    logs = [str(tmp_path / ("c%d.jsonl" % j)) for j in range(2)]
    keep = T._Keep()
    jobs, _, cands = make_jobs(n_jobs, n, keep)
    clients = make_clients(2, logs, keep)
    with pytest.raises(L.CtError) as e:
        L.ct_test_run_clients(clients, jobs, hooks(delay_us=300, stop_after=23))
    assert e.value.code == L.CT_E_STOPPED
    first = T.read_logs(logs)
    n_first = sum(len(v) for v in first["cands"].values())
    assert 23 <= n_first < n_jobs * n and first["duplicates"] == 0
    # resume: recorded candidates are skipped; finished jobs are not run again
    rec = T.resume_state(first, {100 + i: cands for i in range(n_jobs)})
    todo = [i for i in range(n_jobs) if 100 + i not in first["jobs"]]
    keep2 = T._Keep()
    jobs2 = (L.ct_tune_job * len(todo))()
    for k, i in enumerate(todo):
        T.fill_job(jobs2[k], OP, 100 + i, 1, 1, 1, cands, 4, keep2, recorded=rec.get(100 + i))
    clients2 = make_clients(2, logs, keep2)
    L.ct_test_run_clients(clients2, jobs2, hooks())
    assert sum(c.n_measured for c in clients2) == n_jobs * n - n_first
    final = T.read_logs(logs)
    assert final["duplicates"] == 0
    assert all(len(final["cands"][100 + i]) == n for i in range(n_jobs))
    assert set(final["jobs"]) == {100 + i for i in range(n_jobs)}
    # the resumed selection matches an uninterrupted run's
    keep3 = T._Keep()
    jobs3, _, _ = make_jobs(n_jobs, n, keep3)
    L.ct_test_run_clients(make_clients(2), jobs3, hooks())
    for i in range(n_jobs):
        assert final["jobs"][100 + i]["winner_pos"] == jobs3[i].winner_pos


def test_resume_rejects_a_log_of_another_candidate_list(tmp_path):
    logs = [str(tmp_path / "c0.jsonl")]
    keep = T._Keep()
    jobs, _, cands = make_jobs(1, 6, keep)
    L.ct_test_run_clients(make_clients(1, logs, keep), jobs, hooks())
    other = L.ct_sample(OP, 1, 1, 0, 6)
    assert any(L.schedule_tuple(a) != L.schedule_tuple(b) for a, b in zip(cands, other))
    with pytest.raises(ValueError):
        T.resume_state(T.read_logs(logs), {100: other})


def test_unwritable_log_is_a_call_error(tmp_path):
    keep = T._Keep()
    jobs, _, _ = make_jobs(1, 4, keep)
    clients = make_clients(1, [str(tmp_path / "no" / "such" / "dir.jsonl")], keep)
    with pytest.raises(L.CtError) as e:
        L.ct_test_run_clients(clients, jobs, hooks())
    assert e.value.code == L.CT_E_ARG


# ---------------------------------------------------------------- grid size
@pytest.mark.parametrize("name", ["r18.2", "r18.3", "dw1", "pw3"])
def test_grid_size_counts_the_valid_schedules_of_each_family(name):
    op, _, _ = T.find_layer(name)
    space = L.ct_valid_space(op)
    for fam in (1, 2, 3, 4):
        n = L.ct_grid_size(op, fam)
        assert n == sum(1 for s in space if s.family == fam)


def test_empty_and_all_failed_jobs_have_no_winner_and_the_rest_finish():
    # job 0 has no candidates; job 1 resumes a run whose candidates all timed
    # out (every one recorded, none measured again); jobs 2 and 3 are ordinary
    keep = T._Keep()
    cands = L.ct_sample(OP, 0, 1, 0, 12)
    jobs = (L.ct_tune_job * 4)()
    T.fill_job(jobs[0], OP, 100, 1, 1, 1, [], 4, keep)
    T.fill_job(jobs[1], OP, 101, 1, 1, 1, cands, 4, keep,
               recorded={p: (float("inf"), L.S_TIMEOUT) for p in range(12)})
    T.fill_job(jobs[2], OP, 102, 1, 1, 1, cands, 4, keep)
    T.fill_job(jobs[3], OP, 103, 1, 1, 1, cands, 4, keep)
    clients = make_clients(2)
    owner = L.ct_test_run_clients(clients, jobs, hooks(delay_us=100))
    assert (owner >= 0).all()
    assert [jobs[i].rc for i in range(4)] == [0, 0, 0, 0]
    assert jobs[0].winner_pos == -1 and jobs[0].n_top == 0 and jobs[0].winner_lat_us == float("inf")
    assert jobs[1].winner_pos == -1 and jobs[1].n_top == 0 and jobs[1].winner_lat_us == float("inf")
    assert jobs[2].winner_pos >= 0 and jobs[3].winner_pos >= 0
    assert sum(c.n_measured for c in clients) == 24
    assert all(c.rc == 0 for c in clients)


def test_no_jobs_leaves_the_clients_idle():
    clients = make_clients(3)
    owner = L.ct_test_run_clients(clients, (L.ct_tune_job * 0)(), hooks())
    assert owner.size == 0
    assert all(c.rc == 0 and c.n_measured == 0 for c in clients)
