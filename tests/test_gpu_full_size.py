"""Whole-batch parity of the full-size workloads against the fp64 oracle.

For every sequence of each batch the GPU prediction is compared with the
oracle's (stored by tests/golden/make_oracle_preds.py, which runs only the
oracle on the same seeded inputs; the file's SHA-256 of the packed batch must
match the batch generated here). Final hidden states are compared with the
oracle evaluated here: on every sequence of the 64-sequence BERT-base batch,
and on sequences spread over the length distribution elsewhere (for the
XLM-R-large shape one per length decile, the longest, 2048-token-capped
sequences included). The selection is checked end to end on each batch (the
GPU's chosen set against the oracle select on the oracle's predictions,
asserted equal whenever the oracle's gap at the cut exceeds twice the largest
prediction error) and bit-exact on the GPU's own predictions.

Bars as in test_gpu_predict.py. Every measured margin is recorded for the
run's summary (tests/parity_log.py).
"""
import numpy as np
import pytest

import oracle
from paper_2505_09142_amd.device import upload_batch
from tests.golden.make_oracle_preds import digest, load
from tests.gpu_util import note
from tests.parity_log import record
from tests.test_gpu_predict import (HIDDEN_ATOL, PRED_RTOL, Y_RTOL, check_selection, e2e_selection, predictor,
                                    rel_err, y_rel)
from workloads import W_BERT_B64, W_BERT_B64_HEAD8, W_BERT_B256_ROUNDS, W_XLMR_B128, make_batch
from workloads.gen import RoundStream

pytestmark = pytest.mark.gpu


def _golden(stem, b):
    rec = load(stem)
    assert rec["n_seqs"] == b.n and rec["total_tokens"] == b.total
    assert rec["token_ids_sha256"] == digest(b.token_ids) and rec["cu_seqlens_sha256"] == digest(b.cu_seqlens), \
        "the seeded generator no longer produces the batch the stored oracle values were computed on"
    return rec["pred"]


def _run(pr, b, want_hidden):
    ids, cu, arr = upload_batch(b)
    pred, hid = pr.predict(ids, cu, b.max_seqlen, want_hidden=want_hidden)
    st, bits = pr.status()
    assert st == 0, (st, bits)
    return pred.cpu().numpy(), (hid.cpu().numpy() if hid is not None else None), arr


def _hidden_err(W, shape, b, hid, seqs):
    """Largest |H_gpu - H_oracle| over the given sequences, evaluated by the oracle here."""
    ref_p, ref_h = oracle.oracle_forward(b.token_ids, b.cu_seqlens, W.master, shape, seqs=seqs)
    worst = 0.0
    for s in seqs:
        a, e = b.cu_seqlens[s], b.cu_seqlens[s + 1]
        err = float(np.abs(hid[a:e] - ref_h[a:e]).max())
        worst = max(worst, err)
        assert err <= HIDDEN_ATOL, (s, e - a, err)
    return worst, ref_p


def _check_preds(w, pred, ref, what):
    assert np.all(np.isfinite(pred))
    perr = float(rel_err(pred, ref).max())
    yerr = y_rel(pred, ref, w.shape)
    note(f"{what}: pred max-rel {perr:.3e} over all {len(ref)} sequences, y rel {yerr:.3e}")
    assert perr <= PRED_RTOL and yerr <= Y_RTOL
    return perr, yerr


def test_bert_base_b64_whole_batch():
    """Every sequence: predictions, final hidden states, selection (the benchmark's batch)."""
    w = W_BERT_B64
    W, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    note(f"{w.name}: GPU whole batch, oracle on all {b.n} sequences ({b.total} tokens)")
    pred, hid, d_arr = _run(pr, b, True)
    ref = _golden(w.name, b)
    perr, yerr = _check_preds(w, pred, ref, w.name)
    herr, live = _hidden_err(W, w.shape, b, hid, list(range(b.n)))
    # the oracle run here and the stored values agree (same arithmetic, other BLAS threading)
    assert np.abs(live - ref).max() <= 1e-9 * np.abs(ref).max()
    note(f"{w.name}: hidden max-abs {herr:.3e} over all sequences")
    check_selection(pr, pred, d_arr, b.arrival_seq, w.batch_cap)
    sel = e2e_selection(pred, ref, b.arrival_seq, w.batch_cap)
    note(f"{w.name}: selection gap {sel['gap']:.3f} vs 2 x err {2 * sel['max_err']:.3f}")
    record(w.name, seqs=f"all {b.n}", hidden=herr, pred_rel=perr, y_rel=yerr, **sel)


@pytest.mark.parametrize("rnd", [0, 49, 99])
def test_b256_rounds_whole_batch(rnd):
    """Rounds 0, 49 and 99 of the 256-sequence, 100-round workload: every prediction against the
    oracle, hidden states on the shortest, the longest and a random sequence."""
    w = W_BERT_B256_ROUNDS
    W, pr = predictor(w.shape, w.weight_seed)
    b = RoundStream(w).batch(rnd)
    note(f"{w.name} round {rnd}: GPU whole batch ({b.total} tokens), stored oracle predictions")
    pred, hid, d_arr = _run(pr, b, True)
    ref = _golden(f"{w.name}_r{rnd}", b)
    perr, yerr = _check_preds(w, pred, ref, f"{w.name} round {rnd}")
    rng = np.random.default_rng(rnd)
    seqs = sorted({int(np.argmin(b.lengths)), int(np.argmax(b.lengths)), int(rng.integers(b.n))})
    herr, live = _hidden_err(W, w.shape, b, hid, seqs)
    assert np.abs(live[seqs] - ref[seqs]).max() <= 1e-9 * np.abs(ref).max()
    check_selection(pr, pred, d_arr, b.arrival_seq, w.batch_cap)
    sel = e2e_selection(pred, ref, b.arrival_seq, w.batch_cap)
    note(f"{w.name} round {rnd}: hidden {herr:.3e}; selection gap {sel['gap']:.3f} vs 2 x err "
         f"{2 * sel['max_err']:.3f}")
    record(f"{w.name} round {rnd}", seqs=f"pred all {b.n}, hidden {len(seqs)}", hidden=herr, pred_rel=perr,
           y_rel=yerr, **sel)


def _decile_sample(lengths):
    """One sequence at each length decile (sorted order), the longest included."""
    order = np.argsort(lengths, kind="stable")
    at = np.unique(np.round(np.linspace(0, len(lengths) - 1, 11)).astype(int))
    return [int(order[i]) for i in at]


@pytest.mark.parametrize("part", [0, 1])
def test_xlmr_large_whole_batch(part):
    """Every prediction against the oracle; hidden states on one sequence per length decile (the
    shorter half in part 0, the longer half, with a 2048-token sequence, in part 1)."""
    w = W_XLMR_B128
    W, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    pred, hid, d_arr = _run(pr, b, True)
    ref = _golden(w.name, b)
    sample = _decile_sample(b.lengths)
    seqs = sample[:6] if part == 0 else sample[6:]
    lens = [int(b.lengths[s]) for s in seqs]
    if part == 1:
        assert max(lens) == w.max_len, "the longest sampled sequence is capped at the position table"
    note(f"{w.name} part {part}: GPU whole batch, oracle hidden states of sequences of length {lens}")
    perr, yerr = _check_preds(w, pred, ref, w.name)
    herr, live = _hidden_err(W, w.shape, b, hid, seqs)
    assert np.abs(live[seqs] - ref[seqs]).max() <= 1e-9 * np.abs(ref).max()
    check_selection(pr, pred, d_arr, b.arrival_seq, w.batch_cap)
    sel = e2e_selection(pred, ref, b.arrival_seq, w.batch_cap)
    note(f"{w.name}: hidden {herr:.3e}; selection gap {sel['gap']:.3f} vs 2 x err {2 * sel['max_err']:.3f}")
    record(f"{w.name} (hidden lengths {min(lens)}-{max(lens)})", seqs=f"pred all {b.n}, hidden {len(seqs)}",
           hidden=herr, pred_rel=perr, y_rel=yerr, **sel)


def test_bert_base_head8_whole_batch():
    """The paper's eight-layer, width-1024 head on mean pooling: every prediction against the
    oracle, hidden states on the shortest, the longest and a random sequence."""
    w = W_BERT_B64_HEAD8
    W, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    note(f"{w.name}: GPU whole batch, stored oracle predictions")
    pred, hid, d_arr = _run(pr, b, True)
    ref = _golden(w.name, b)
    perr, yerr = _check_preds(w, pred, ref, w.name)
    seqs = sorted({int(np.argmin(b.lengths)), int(np.argmax(b.lengths)), 17})
    herr, live = _hidden_err(W, w.shape, b, hid, seqs)
    assert np.abs(live[seqs] - ref[seqs]).max() <= 1e-9 * np.abs(ref).max()
    check_selection(pr, pred, d_arr, b.arrival_seq, w.batch_cap)
    sel = e2e_selection(pred, ref, b.arrival_seq, w.batch_cap)
    record(w.name, seqs=f"pred all {b.n}, hidden {len(seqs)}", hidden=herr, pred_rel=perr, y_rel=yerr, **sel)


@pytest.mark.parametrize("w", [W_BERT_B64, W_BERT_B64_HEAD8], ids=lambda w: w.name)
def test_predictions_without_hidden_output_match(w):
    """The benchmark calls predict without a hidden-state output (CLS pooling then runs the last
    layer on the CLS rows only): those predictions meet the same bars against the oracle."""
    W, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    note(f"{w.name}: predictions only (no hidden output), every sequence")
    pred, _, d_arr = _run(pr, b, False)
    ref = _golden(w.name, b)
    perr, yerr = _check_preds(w, pred, ref, f"{w.name} (no hidden output)")
    sel = e2e_selection(pred, ref, b.arrival_seq, w.batch_cap)
    record(f"{w.name} (predict only)", seqs=f"pred all {b.n}", pred_rel=perr, y_rel=yerr, **sel)
