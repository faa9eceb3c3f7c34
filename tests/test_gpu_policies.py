"""Scheduler variants on the device job table (FCFS, SJF, ISRTF with a stand-in predictor of
the paper's accuracy, aging, preemption cost) against the oracle simulator.

* elis_jobs_select_aged ranks candidates exactly as the oracle select ranks the
  oracle's aged keys (fp64 evaluation, one rounding to fp32), bit for bit, with
  ties, NaN, signed zeros and infinities, up to 10000 active jobs (the
  device-wide radix path).
* The loop on the device reproduces the oracle simulator's trajectory round by
  round (times, batches, re-prefilled jobs, window lengths) and its finish
  times and preemption counts exactly, for every policy with and without aging
  and re-prefill cost, on the 200-request Gamma-arrival study stream.
* With the encoder as the predictor, aging and re-prefill cost on the device
  table also follow the oracle (predictions replayed into the oracle).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_09142_amd import _elis as E
from paper_2505_09142_amd.device import JobTable
from paper_2505_09142_amd.driver import DeviceRoundDriver
from paper_2505_09142_amd.scheduler import run_schedule
from tests.gpu_util import note
from tests.test_gpu_predict import predictor
from workloads import POLICY_STUDY, S_ISRTF, accuracy_model_keys, make_policy_requests, make_requests

pytestmark = pytest.mark.gpu


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).cuda()


@pytest.mark.parametrize("a", [1, 700, 10000])
def test_aged_select_matches_oracle(a):
    rng = np.random.default_rng(100 + a)
    J = max(2 * a, 64)
    tab = JobTable(J, 8)
    slots = rng.permutation(J)[:a].astype(np.int32)
    arrival = rng.permutation(a).astype(np.int64)
    key = rng.integers(0, 40, size=a).astype(np.float32)                 # many ties before aging
    key[rng.random(a) < 0.01] = np.nan
    key[rng.random(a) < 0.01] = -0.0
    key[rng.random(a) < 0.005] = np.inf
    wait = (rng.integers(0, 8, size=a) * 0.25).astype(np.float32)         # exact multiples: ties after aging
    frac = rng.random(a) < 0.2
    wait[frac] = rng.random(int(frac.sum())).astype(np.float32)   # and arbitrary fractions
    tab.start(_dev(slots, np.int32), _dev(arrival, np.int64))
    tab.store_pred(_dev(slots, np.int32), _dev(key, np.float32))
    for aging in (0.0, 4.0, 500.0, -3.5):
        aged = oracle.aged_keys(key, wait, aging)
        for cap in (1, 32, min(a, 8192)):
            note(f"aged select a={a} aging={aging} cap={cap}")
            out = torch.full((max(1, cap),), -1, dtype=torch.int32, device="cuda")
            cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
            tab.select(_dev(slots, np.int32), cap, out, cnt, wait=_dev(wait, np.float32), aging=aging)
            torch.cuda.synchronize()
            m = int(cnt.item())
            assert m == min(cap, a)
            exp = slots[oracle.oracle_select(aged, arrival, cap)]
            assert np.array_equal(out.cpu().numpy()[:m], exp), (a, aging, cap)
    st, bits = tab.status()
    assert st == E.ELIS_OK and bits == 0


def _compare(got, ref):
    assert len(got.rounds) == len(ref.rounds)
    for i, (a, b) in enumerate(zip(got.rounds, ref.rounds)):
        assert a.t == b.t, i
        assert list(a.rescored) == list(b.rescored) and list(a.candidates) == list(b.candidates), i
        assert list(a.chosen) == list(b.selected), i
        assert list(a.resumed) == list(b.resumed) and a.prefill_s == b.prefill_s, i
        assert a.steps == b.window_steps, i
    assert np.array_equal(got.finish_t, ref.finish_t)
    assert np.array_equal(got.preemptions, ref.preemptions)
    assert np.array_equal(got.generated, ref.generated)


@pytest.mark.parametrize("policy", ["fcfs", "sjf", "isrtf"])
@pytest.mark.parametrize("aging,prefill", [(0.0, 0.0), (POLICY_STUDY.aging, 0.0),
                                           (POLICY_STUDY.aging, POLICY_STUDY.prefill_cost_s)])
def test_policy_loop_matches_oracle(policy, aging, prefill):
    st = POLICY_STUDY
    req = make_policy_requests(st, 4, 3.0, 0)
    rem = np.array([len(r) for r in req.response])

    def key_fn(jobs, gen):
        jobs = np.asarray(jobs)
        return accuracy_model_keys(st.data_seed, jobs, gen[jobs], rem[jobs] - gen[jobs], st.accuracy_mae)

    note(f"policy loop {policy} aging={aging} prefill={prefill}")
    drv = DeviceRoundDriver(None, 256, 8)
    got = run_schedule(req.arrival_t, req.prompt, req.response, drv, window=st.window, step_cost=st.step_cost_s,
                       batch_cap=4, policy=policy, key_fn=key_fn if policy == "isrtf" else None, aging=aging,
                       prefill_cost=prefill)
    ref = oracle.simulate(req.arrival_t, req.prompt, req.response, window=st.window, step_cost=st.step_cost_s,
                          batch_cap=4, max_pos=8, policy=policy, aging=aging, prefill_cost=prefill,
                          predict_fn=(lambda todo, inputs, g: key_fn(todo, g)) if policy == "isrtf" else None)
    _compare(got, ref)
    t, bits = drv.table.status()
    assert t == E.ELIS_OK and bits == 0
    note(f"  {len(got.rounds)} rounds, mean JCT {np.mean(got.jct):.2f} s, "
         f"{int(got.preemptions.sum())} preemptions")


def test_encoder_loop_with_aging_and_prefill_matches_oracle():
    s = S_ISRTF
    W, pr = predictor(s.shape, s.weight_seed)
    req = make_requests(s, n=300)
    rounds = 60
    note(f"encoder ISRTF loop with aging and re-prefill cost, {rounds} rounds")
    drv = DeviceRoundDriver(pr, 512, s.shape.max_pos)
    got = run_schedule(req.arrival_t, req.prompt, req.response, drv, window=s.window, step_cost=s.step_cost_s,
                       batch_cap=16, policy="isrtf", aging=POLICY_STUDY.aging,
                       prefill_cost=POLICY_STUDY.prefill_cost_s, max_rounds=rounds)
    replay = iter([r.pred for r in got.rounds if len(r.rescored)])
    ref = oracle.simulate(req.arrival_t, req.prompt, req.response, window=s.window, step_cost=s.step_cost_s,
                          batch_cap=16, max_pos=s.shape.max_pos, policy="isrtf", aging=POLICY_STUDY.aging,
                          prefill_cost=POLICY_STUDY.prefill_cost_s, max_rounds=rounds,
                          predict_fn=lambda todo, inputs, g: next(replay))
    assert len(got.rounds) == len(ref.rounds) == rounds
    for i, (a, b) in enumerate(zip(got.rounds, ref.rounds)):
        assert a.t == b.t and list(a.chosen) == list(b.selected), i
        assert list(a.resumed) == list(b.resumed) and a.steps == b.window_steps, i
    assert sum(len(r.resumed) for r in got.rounds) > 0, "the prefix should exercise a re-prefill"
    t, bits = drv.table.status()
    assert t == E.ELIS_OK and bits == 0
