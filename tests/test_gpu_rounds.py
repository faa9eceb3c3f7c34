"""Multi-round workloads on the GPU path.

* 256 in-flight sequences re-scored for 100 rounds, each growing by one token
  per round: every round's GPU selection is checked bit-exact against the
  oracle select on the same predictions; the oracle encoder spot-checks
  sampled sequences at rounds 0, 49 and 99.
* The one-node ISRTF loop over 4096 synthetic requests, teacher-forced: the
  oracle simulator is the state of record, the GPU driver builds and scores
  the inputs, and every round the GPU selection must equal the oracle
  selection on the same predictions. The oracle encoder spot-checks
  predictions on at least 10 rounds.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_09142_amd.device import upload_batch
from paper_2505_09142_amd.driver import RoundDriver
from tests.gpu_util import note
from tests.test_gpu_predict import HIDDEN_ATOL, PRED_RTOL, predictor, rel_err
from workloads import S_ISRTF, W_BERT_B256_ROUNDS, make_requests
from workloads.gen import RoundStream

pytestmark = pytest.mark.gpu


def test_b256_hundred_rounds():
    w = W_BERT_B256_ROUNDS
    W, pr = predictor(w.shape, w.weight_seed)
    rs = RoundStream(w)
    check = {0: [3, 200], 49: [17, 101], 99: [64, 255]}
    for r in range(w.rounds):
        b = rs.batch(r)
        ids, cu, arr = upload_batch(b)
        pred, hid = pr.predict(ids, cu, b.max_seqlen, want_hidden=r in check)
        p = pred.cpu().numpy()
        idx, cnt = pr.select(pred, arr, w.batch_cap)
        got = idx[:int(cnt.item())].cpu().numpy()
        assert np.array_equal(got, oracle.oracle_select(p, b.arrival_seq, w.batch_cap)), f"round {r}"
        if r in check:
            h = hid.cpu().numpy()
            ref_p, ref_h = oracle.oracle_forward(b.token_ids, b.cu_seqlens, W.master, w.shape, seqs=check[r])
            for s in check[r]:
                a, e = b.cu_seqlens[s], b.cu_seqlens[s + 1]
                herr = np.abs(h[a:e] - ref_h[a:e]).max()
                perr = rel_err(p[s], ref_p[s])
                note(f"round {r} seq {s} len {e - a} T={b.total}: hidden {herr:.3e} pred {perr:.3e}")
                assert herr <= HIDDEN_ATOL and perr <= PRED_RTOL
    st, bits = pr.status()
    assert st == 0, bits


def test_isrtf_loop_teacher_forced():
    s = S_ISRTF
    W, pr = predictor(s.shape, s.weight_seed)
    req = make_requests(s)
    drv = RoundDriver(pr, s.shape.max_pos)
    calls = {"n": 0, "checked": 0}
    mismatches = []

    def predict_fn(job_ids, inputs, g):
        gpu = drv.predict_jobs(job_ids, req.prompt, req.response, g)
        calls["n"] += 1
        if calls["n"] % 40 == 1:
            j = len(job_ids) // 2
            ref_p, _ = oracle.oracle_forward(inputs[j], np.array([0, len(inputs[j])]), W.master, s.shape,
                                             want_hidden=False)
            perr = rel_err(gpu[j], ref_p[0])
            note(f"round {calls['n']}: job {job_ids[j]} len {len(inputs[j])} gpu {gpu[j]:.3f} "
                 f"oracle {ref_p[0]:.3f} rel {perr:.2e}")
            assert perr <= PRED_RTOL
            calls["checked"] += 1
        return gpu

    def select_fn(pred32, arrival, cap):
        exp = oracle.oracle_select(pred32, arrival, cap)
        got = drv.select(pred32, arrival, cap)
        if not np.array_equal(got, exp):
            mismatches.append((calls["n"], got, exp))
        return exp

    res = oracle.simulate(req.arrival_t, req.prompt, req.response, window=s.window, step_cost=s.step_cost_s,
                          batch_cap=s.batch_cap, max_pos=s.shape.max_pos, predict_fn=predict_fn,
                          select_fn=select_fn)
    note(f"ISRTF loop: {len(res.rounds)} rounds, mean JCT {np.nanmean(res.jct):.2f} s, "
         f"max candidates {max(len(r.candidates) for r in res.rounds)}")
    assert not mismatches, mismatches[:3]
    assert calls["checked"] >= 10
    assert np.array_equal(res.generated, [len(x) for x in req.response])
