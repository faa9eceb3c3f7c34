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

from oracle import aged_keys, job_input, simulate


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


# ----------------------------------------------------------------------------- policies, aging, preemption cost

def test_fcfs_policy_runs_in_arrival_order():
    lengths = [7, 2, 11, 4, 9, 3]
    prompts, responses = _jobs(lengths, 1)
    c = 0.5
    res = simulate(np.zeros(6), prompts, responses, window=50, step_cost=c, batch_cap=1, max_pos=64, policy="fcfs")
    # one slot, every job fits one window: jobs finish back to back in arrival order
    np.testing.assert_allclose(res.finish_t, np.cumsum(lengths) * c)
    assert [rr.selected for rr in res.rounds] == [[j] for j in range(6)]


@pytest.mark.parametrize("lengths", [[5, 2, 9, 1], [3, 3, 1, 7, 2], [4, 8, 1, 6, 2, 5]])
def test_sjf_policy_is_optimal_for_simultaneous_arrivals(lengths):
    prompts, responses = _jobs(lengths)
    c = 0.01
    res = simulate(np.zeros(len(lengths)), prompts, responses, window=3, step_cost=c, batch_cap=1, max_pos=64,
                   policy="sjf")
    best = min(np.mean(np.cumsum([lengths[i] for i in order]) * c)
               for order in itertools.permutations(range(len(lengths))))
    assert abs(np.mean(res.jct) - best) < 1e-9


def test_aged_keys_rounding():
    # exact cases: 100 - 500 * fl32(0.1) = 49.99999925..., which rounds to 50 in fp32
    assert aged_keys(np.float32([100.0]), np.float32([0.1]), 500.0)[0] == np.float32(50.0)
    # aging 0 leaves every key (and its sign of zero) unchanged
    k = np.float32([-0.0, 0.0, 3.5, np.inf, -np.inf])
    out = aged_keys(k, np.float32([1, 2, 3, 4, 5]), 0.0)
    assert np.array_equal(out.view(np.uint32), k.view(np.uint32))
    assert np.isnan(aged_keys(np.float32([np.nan]), np.float32([1.0]), 2.0)[0])
    # an fp32 result that needs the fp64 intermediate: 2^24 + 1 is not an fp32 value
    got = aged_keys(np.float32([16777216.0]), np.float32([1.0]), -1.0)[0]
    assert got == np.float32(16777216.0)      # 16777217 rounds to even
    assert aged_keys(np.float32([3e38]), np.float32([1e30]), -1e10)[0] == np.inf


def test_aging_and_preemption_cost_hand_example():
    """Two jobs at t = 0 with 3-token prompts; SJF keys A = 30, B = 20; windows of 10 tokens at
    0.01 s per step; aging 500 tokens/s; re-prefill 0.001 s per token. Worked by hand:
      t=0      keys A 30, B 20                     -> B runs 10 tokens, ends 0.1
      t=0.1    A waited 0.1: 30 - 50 = -20; B 20   -> A runs (first run, free), B preempted
      t=0.2    A 30; B waited 0.1: 20 - 50 = -30   -> B resumes: re-prefill 3 + 10 = 13 tokens
                                                       (0.013 s), finishes at 0.2 + 0.013 + 0.1 = 0.313
      t=0.313  A alone, preempted at 0.2           -> re-prefill 13 tokens, runs to 0.426
      t=0.426  A (ran last, KV kept)               -> finishes at 0.526
    """
    prompts, responses = _jobs([30, 20], 6)
    res = simulate(np.zeros(2), prompts, responses, window=10, step_cost=0.01, batch_cap=1, max_pos=64,
                   policy="sjf", aging=500.0, prefill_cost=0.001)
    assert [rr.selected for rr in res.rounds] == [[1], [0], [1], [0], [0]]
    assert [rr.resumed for rr in res.rounds] == [[], [], [1], [0], []]
    np.testing.assert_allclose([rr.t for rr in res.rounds], [0.0, 0.1, 0.2, 0.313, 0.426], atol=1e-12)
    np.testing.assert_allclose(res.finish_t, [0.526, 0.313], atol=1e-12)
    assert res.preemptions.tolist() == [1, 1]
    np.testing.assert_allclose(res.queue_delay, [0.526 - 0.3, 0.313 - 0.2], atol=1e-12)
    # without aging the short job runs to completion first and nothing is preempted
    plain = simulate(np.zeros(2), prompts, responses, window=10, step_cost=0.01, batch_cap=1, max_pos=64,
                     policy="sjf", prefill_cost=0.001)
    assert [rr.selected for rr in plain.rounds] == [[1], [1], [0], [0], [0]]
    assert plain.preemptions.tolist() == [0, 0]
    np.testing.assert_allclose(plain.finish_t, [0.5, 0.2], atol=1e-12)


@pytest.mark.parametrize("policy", ["fcfs", "sjf", "isrtf"])
def test_conservation_with_aging_and_prefill(policy):
    rng = np.random.default_rng(11)
    lengths = rng.integers(1, 150, size=40)
    prompts, responses = _jobs(lengths, 9)
    arrival = np.sort(rng.uniform(0, 1.5, size=40))
    c, cp = 0.01, 0.0005
    res = simulate(arrival, prompts, responses, window=20, step_cost=c, batch_cap=3, max_pos=64, policy=policy,
                   predict_fn=_true_remaining(responses), aging=30.0, prefill_cost=cp)
    assert np.array_equal(res.generated, lengths)
    assert np.all(res.queue_delay >= -1e-12)
    # preemptions recounted from the trajectory: a job in one batch, unfinished, absent from the next
    recount = np.zeros(len(lengths), dtype=np.int64)
    for a, b in zip(res.rounds, res.rounds[1:]):
        for j in a.selected:
            if j in b.candidates and j not in b.selected:
                recount[j] += 1
    assert np.array_equal(recount, res.preemptions)
    # every re-prefill is paid by a job preempted earlier, and costs at least its prompt
    assert sum(len(rr.resumed) for rr in res.rounds) <= res.preemptions.sum()
    for rr in res.rounds:
        if rr.resumed:
            assert rr.prefill_s >= cp * sum(len(prompts[j]) for j in rr.resumed) - 1e-15
        else:
            assert rr.prefill_s == 0.0
    # the clock only moves by window lengths (and jumps to the next arrival when idle)
    for a, b in zip(res.rounds, res.rounds[1:]):
        assert b.t >= a.t + a.prefill_s + a.window_steps * c - 1e-12


def test_aging_zero_equals_plain_select():
    rng = np.random.default_rng(2)
    lengths = rng.integers(5, 80, size=25)
    prompts, responses = _jobs(lengths, 4)
    arrival = np.sort(rng.uniform(0, 0.5, size=25))
    a = simulate(arrival, prompts, responses, window=10, step_cost=0.01, batch_cap=2, max_pos=64, policy="sjf")
    b = simulate(arrival, prompts, responses, window=10, step_cost=0.01, batch_cap=2, max_pos=64, policy="sjf",
                 aging=0.0, prefill_cost=0.0)
    assert [r.selected for r in a.rounds] == [r.selected for r in b.rounds]
    assert np.array_equal(a.finish_t, b.finish_t)


# ----------------------------------------------------------------------------- window end and re-scoring rules

def test_first_finish_window_end_hand_example():
    """end_rule "first" (the alternative reading of the window end, Sec. 4.1): the window ends when
    the first selected job stops. Three jobs at t = 0 with 4, 15 and 6 response tokens, FCFS keys,
    two slots, windows of 10 tokens at 0.01 s per step. Worked by hand:
      t=0     A, B run; A has 4 left, B 10 of its window -> the window lasts 4 steps:
              A finishes at 0.04, B is credited 4 tokens (not its 10)
      t=0.04  B (11 left), C (6 left) run          -> 6 steps: C finishes at 0.10, B at 10 tokens
      t=0.10  B alone, 5 left                      -> finishes at 0.15
    With end_rule "all" the first window lasts 10 steps (B reaches 10 tokens at 0.10); then B and C
    run together, B finishing at 0.15 and C at 0.16.
    """
    prompts, responses = _jobs([4, 15, 6], 12)
    kw = dict(window=10, step_cost=0.01, batch_cap=2, max_pos=64, policy="fcfs")
    first = simulate(np.zeros(3), prompts, responses, end_rule="first", **kw)
    assert [rr.selected for rr in first.rounds] == [[0, 1], [1, 2], [1]]
    assert [rr.window_steps for rr in first.rounds] == [4, 6, 5]
    np.testing.assert_allclose([rr.t for rr in first.rounds], [0.0, 0.04, 0.10], atol=1e-12)
    np.testing.assert_allclose(first.finish_t, [0.04, 0.15, 0.10], atol=1e-12)
    assert first.generated.tolist() == [4, 15, 6]
    every = simulate(np.zeros(3), prompts, responses, end_rule="all", **kw)
    assert [rr.selected for rr in every.rounds] == [[0, 1], [1, 2]]
    assert [rr.window_steps for rr in every.rounds] == [10, 6]
    np.testing.assert_allclose(every.finish_t, [0.04, 0.15, 0.16], atol=1e-12)


def test_first_finish_conservation():
    rng = np.random.default_rng(21)
    lengths = rng.integers(1, 90, size=30)
    prompts, responses = _jobs(lengths, 13)
    arrival = np.sort(rng.uniform(0, 1.0, size=30))
    res = simulate(arrival, prompts, responses, window=25, step_cost=0.01, batch_cap=4, max_pos=64,
                   predict_fn=_true_remaining(responses), end_rule="first")
    assert np.array_equal(res.generated, lengths)
    for rr in res.rounds:
        # the window is the shortest of the chosen jobs' budgets min(K, tokens left)
        assert 1 <= rr.window_steps <= 25
    assert np.all(res.jct >= lengths * 0.01 - 1e-12)


def _counting_predictor(base, drop):
    """A predictor whose key for job j falls by drop[j] each time j is scored: its output depends on
    how often a job was re-scored, so re-scoring rules become visible in the trajectory."""
    calls = {}

    def fn(ids, inputs, g):
        out = []
        for j in ids:
            c = calls.get(j, 0)
            calls[j] = c + 1
            out.append(float(base[j] - drop[j] * c))
        return out
    return fn


def test_rescore_all_rekeys_every_candidate_hand_example():
    """rescore "all" (reading of cfg5's re-score-all) gives every admitted unfinished job a fresh key
    each round; "pool" (Alg. 1) only the new arrivals and the jobs that ran. Two jobs of 20 tokens at
    t = 0, one slot, windows of 10; a predictor whose key for A is 50 - 30 c and for B 60 - 50 c after
    c earlier scorings. Worked by hand:
      pool: t=0 A 50, B 60 -> A;  A re-scored 20, B keeps 60 -> A (finishes 0.2);  B 60 -> B;  B 10 -> B
      all:  t=0 A 50, B 60 -> A;  A 20, B 10 -> B;  A -10, B -40 -> B (finishes 0.3);  A -40 -> A
    """
    prompts, responses = _jobs([20, 20], 14)
    kw = dict(window=10, step_cost=0.01, batch_cap=1, max_pos=64)
    pool = simulate(np.zeros(2), prompts, responses, predict_fn=_counting_predictor([50, 60], [30, 50]),
                    rescore="pool", **kw)
    assert [rr.selected for rr in pool.rounds] == [[0], [0], [1], [1]]
    assert [rr.rescored for rr in pool.rounds] == [[0, 1], [0], [], [1]]
    np.testing.assert_allclose(pool.finish_t, [0.2, 0.4], atol=1e-12)
    every = simulate(np.zeros(2), prompts, responses, predict_fn=_counting_predictor([50, 60], [30, 50]),
                     rescore="all", **kw)
    assert [rr.selected for rr in every.rounds] == [[0], [1], [1], [0]]
    assert [rr.rescored for rr in every.rounds] == [[0, 1], [0, 1], [0, 1], [0]]
    np.testing.assert_allclose([rr.pred.tolist() for rr in every.rounds[:3]], [[50, 60], [20, 10], [-10, -40]])
    np.testing.assert_allclose(every.finish_t, [0.4, 0.3], atol=1e-12)
    for rr in every.rounds:
        assert rr.rescored == rr.candidates


@pytest.mark.parametrize("end_rule", ["all", "first"])
def test_rescore_all_equals_pool_for_a_deterministic_predictor(end_rule):
    """A predictor that is a function of the job's input alone gives an unchanged job the key it
    already has, so re-scoring every job reproduces the Job-Pool trajectory exactly (reading 15)."""
    rng = np.random.default_rng(31)
    lengths = rng.integers(1, 200, size=60)
    prompts, responses = _jobs(lengths, 15)
    arrival = np.sort(rng.uniform(0, 2.0, size=60))

    def fn(ids, inputs, g):
        # depends on the input tokens only (length and content)
        return [float((len(x) * 7919 + int(np.sum(x.astype(np.int64) * np.arange(1, len(x) + 1)))) % 997)
                for x in inputs]

    kw = dict(window=20, step_cost=0.01, batch_cap=3, max_pos=32, predict_fn=fn, end_rule=end_rule)
    pool = simulate(arrival, prompts, responses, rescore="pool", **kw)
    every = simulate(arrival, prompts, responses, rescore="all", **kw)
    assert len(pool.rounds) == len(every.rounds)
    for a, b in zip(pool.rounds, every.rounds):
        assert a.t == b.t and a.selected == b.selected and a.window_steps == b.window_steps
        assert np.array_equal(a.keys, b.keys)
        assert set(a.rescored) <= set(b.rescored) and b.rescored == b.candidates
    assert np.array_equal(pool.finish_t, every.finish_t)
