"""The stored whole-batch oracle predictions (tests/golden/oracle_preds_*.json) against the oracle.

Each file must describe the batch the seeded generator produces today (sizes and
SHA-256 of the packed ids and cu_seqlens), hold a finite prediction per
sequence, and agree with the oracle re-run here on its two shortest sequences
(the BERT-base-shaped batches; the XLM-R-large-shaped one only by its batch
digest, its weights take half a minute to draw). Up to BLAS threading the
arithmetic is the same, so the agreement is to ~1e-12.
"""
import numpy as np
import pytest

import oracle
from tests.golden.make_oracle_preds import BATCHES, batch_of, digest, load
from workloads import make_weights


@pytest.mark.parametrize("stem,w,rnd", BATCHES, ids=[b[0] for b in BATCHES])
def test_stored_oracle_predictions(stem, w, rnd):
    rec = load(stem)
    b = batch_of(w, rnd)
    assert rec["workload"] == w.name and rec["round"] == rnd
    assert rec["n_seqs"] == b.n and rec["total_tokens"] == b.total
    assert rec["token_ids_sha256"] == digest(b.token_ids)
    assert rec["cu_seqlens_sha256"] == digest(b.cu_seqlens)
    pred = rec["pred"]
    assert pred.shape == (b.n,) and np.all(np.isfinite(pred))
    if w.shape.d_model > 768:
        return
    W = make_weights(w.shape, w.weight_seed)
    seqs = [int(s) for s in np.argsort(b.lengths, kind="stable")[:2]]
    p, _ = oracle.oracle_forward(b.token_ids, b.cu_seqlens, W.master, w.shape, want_hidden=False, seqs=seqs)
    assert np.abs(p[seqs] - pred[seqs]).max() <= 1e-9 * np.abs(pred).max()
