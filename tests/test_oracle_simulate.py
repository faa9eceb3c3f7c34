"""Pins of the one-node scheduling-loop oracle.

* SJF optimality (a textbook fact the paper relies on, Sec. 2.2): with all jobs
  present at t = 0, one slot, one-token windows and exact remaining-length
  predictions, the mean JCT equals the minimum over all job orders, found by
  brute force;
* equal predictions reduce the loop to FCFS (Sec. 6.1 baseline), whose
  completion times have a closed form;
* conservation: every job generates exactly its response length; JCT is at
  least R times the step cost;
* a forced preemption: a shorter arrival displaces a running long job.
"""
import itertools

import numpy as np
import pytest

from oracle import job_input, simulate


def _true_remaining(responses):
    R = np.array([len(r) for r in responses])

    def fn(ids, inputs, g):
        return [float(R[j] - g[j]) for j in ids]
    return fn


def _const(ids, inputs, g):
    return [5.0] * len(ids)


def _jobs(lengths, seed=0):
    rng = np.random.default_rng(seed)
    prompts = [rng.integers(1, 50, size=3).astype(np.int32) for _ in lengths]
    responses = [rng.integers(1, 50, size=int(L)).astype(np.int32) for L in lengths]
    return prompts, responses


@pytest.mark.parametrize("lengths", [[5, 2, 9, 1], [3, 3, 1, 7, 2], [4, 8, 1, 6, 2, 5]])
def test_srtf_with_exact_predictions_is_sjf_optimal(lengths):
    prompts, responses = _jobs(lengths)
    c = 0.01
    res = simulate(np.zeros(len(lengths)), prompts, responses, window=1, step_cost=c, batch_cap=1,
                   max_pos=64, predict_fn=_true_remaining(responses))
    best = min(np.mean(np.cumsum([lengths[i] for i in order]) * c)
               for order in itertools.permutations(range(len(lengths))))
    assert abs(np.mean(res.jct) - best) < 1e-9


@pytest.mark.parametrize("window,cap", [(1, 1), (50, 1), (3, 2)])
def test_equal_predictions_give_fcfs(window, cap):
    lengths = [7, 2, 11, 4, 9, 3]
    prompts, responses = _jobs(lengths, 1)
    c = 0.5
    res = simulate(np.zeros(6), prompts, responses, window=window, step_cost=c, batch_cap=cap,
                   max_pos=64, predict_fn=_const)
    for rr in res.rounds:
        assert rr.selected == rr.candidates[:cap]
    if cap == 1:
        # one slot: jobs run to completion in arrival order
        np.testing.assert_allclose(res.finish_t, np.cumsum(lengths) * c)


def test_conservation_and_lower_bound():
    rng = np.random.default_rng(5)
    lengths = rng.integers(1, 120, size=30)
    prompts, responses = _jobs(lengths, 2)
    arrival = np.sort(rng.uniform(0, 2.0, size=30))
    res = simulate(arrival, prompts, responses, window=50, step_cost=0.01, batch_cap=4, max_pos=64,
                   predict_fn=_true_remaining(responses))
    assert np.array_equal(res.generated, lengths)
    assert np.all(res.jct >= lengths * 0.01 - 1e-12)
    assert np.all(res.first_run_t >= arrival - 1e-12)
    # every round's selection is within the cap and drawn from the candidates
    for rr in res.rounds:
        assert len(rr.selected) == min(4, len(rr.candidates))
        assert set(rr.selected) <= set(rr.candidates)


def test_short_arrival_preempts_long_job():
    # job 0 (100 tokens) starts alone; job 1 (10 tokens) arrives during its first window
    prompts, responses = _jobs([100, 10], 3)
    res = simulate(np.array([0.0, 0.05]), prompts, responses, window=10, step_cost=0.01, batch_cap=1,
                   max_pos=64, predict_fn=_true_remaining(responses))
    sel = [rr.selected for rr in res.rounds]
    assert sel[0] == [0]
    assert sel[1] == [1]            # job 0 (90 left) is preempted by job 1 (10 left)
    assert res.finish_t[1] == pytest.approx(0.2)
    assert res.finish_t[0] == pytest.approx(1.1)


def test_pool_rescoring_only_touches_changed_jobs():
    prompts, responses = _jobs([30, 30, 30], 4)
    res = simulate(np.zeros(3), prompts, responses, window=10, step_cost=0.01, batch_cap=1, max_pos=64,
                   predict_fn=_true_remaining(responses))
    assert res.rounds[0].rescored == [0, 1, 2]
    for prev, cur in zip(res.rounds, res.rounds[1:]):
        assert cur.rescored == sorted(j for j in prev.selected if j in cur.candidates)


def test_job_input_truncation():
    prompt = np.arange(1, 6, dtype=np.int32)
    resp = np.arange(100, 110, dtype=np.int32)
    assert job_input(prompt, resp, 3, 64).tolist() == [1, 2, 3, 4, 5, 100, 101, 102]
    # 15 tokens, keep the first and the last 5
    assert job_input(prompt, resp, 10, 6).tolist() == [1, 105, 106, 107, 108, 109]
