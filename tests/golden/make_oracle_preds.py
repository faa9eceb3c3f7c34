"""Write the fp64 oracle's predictions for every sequence of the full-size batches.

    python -m tests.golden.make_oracle_preds [--procs 8] [names ...]

The full-size parity tests compare the GPU's predictions for a whole batch (and
its selection, end to end) with these values; running the oracle over every
sequence of those batches takes minutes to tens of minutes on a CPU, too long
for a test run. This script calls only the oracle (``oracle.oracle_forward``)
and the seeded input generators (``workloads``); nothing it stores comes from
the GPU path. Each file also records a SHA-256 of the packed token ids and
cu_seqlens it was computed from, so a test can confirm that the generator still
produces the same batch.

Batches: the 64 BERT-base sequences, the 256 sequences of the 100-round
workload at rounds 0, 49 and 99, the 128 XLM-R-large-shaped sequences, and the
64 sequences of the BERT-base predictor with the eight-layer head.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import json
import multiprocessing as mp
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from workloads import (W_BERT_B64, W_BERT_B64_HEAD8, W_BERT_B256_ROUNDS, W_XLMR_B128, make_batch,  # noqa: E402
                       make_weights)
from workloads.gen import RoundStream  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))

# (file stem, workload, round or None)
BATCHES = [
    ("bert_base_b64", W_BERT_B64, None),
    ("bert_base_b256_x100_r0", W_BERT_B256_ROUNDS, 0),
    ("bert_base_b256_x100_r49", W_BERT_B256_ROUNDS, 49),
    ("bert_base_b256_x100_r99", W_BERT_B256_ROUNDS, 99),
    ("xlmr_large_b128", W_XLMR_B128, None),
    ("bert_base_head8_b64", W_BERT_B64_HEAD8, None),
]


def batch_of(w, rnd):
    return make_batch(w) if rnd is None else RoundStream(w).batch(rnd)


def digest(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a, dtype=np.int32).tobytes()).hexdigest()


def path_of(stem: str) -> str:
    return os.path.join(HERE, f"oracle_preds_{stem}.json")


_job = {}


def _init():
    # one BLAS thread per worker: the workers split the sequences instead
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except ImportError:
        pass


def _one(s: int) -> tuple:
    b = _job["b"]
    p, _ = oracle.oracle_forward(b.token_ids, b.cu_seqlens, _job["W"].master, _job["shape"], want_hidden=False,
                                 seqs=[s])
    return s, float(p[s])


def compute(stem: str, w, rnd, procs: int) -> dict:
    b = batch_of(w, rnd)
    # weights and batch are built once here; the forked workers share them
    _job.update(W=make_weights(w.shape, w.weight_seed), b=b, shape=w.shape)
    order = [int(s) for s in np.argsort(-b.lengths, kind="stable")]  # longest first: balanced workers
    t0 = time.time()
    pred = np.full(b.n, np.nan)
    ctx = mp.get_context("fork")
    with cf.ProcessPoolExecutor(procs, mp_context=ctx, initializer=_init) as ex:
        for i, (s, v) in enumerate(ex.map(_one, order)):
            pred[s] = v
            if (i + 1) % 16 == 0:
                print(f"  {stem}: {i + 1}/{b.n} sequences, {time.time() - t0:.0f} s", flush=True)
    assert np.all(np.isfinite(pred))
    return {
        "what": "fp64 oracle predictions (out_shift + out_scale * head output) for every sequence",
        "writer": "tests/golden/make_oracle_preds.py (oracle.oracle_forward on workloads' seeded inputs)",
        "workload": w.name,
        "round": rnd,
        "n_seqs": int(b.n),
        "total_tokens": int(b.total),
        "token_ids_sha256": digest(b.token_ids),
        "cu_seqlens_sha256": digest(b.cu_seqlens),
        "oracle_seconds": round(time.time() - t0, 1),
        "pred": [repr(float(v)) for v in pred],
    }


def load(stem: str) -> dict:
    """The stored record, with ``pred`` as a float64 array."""
    with open(path_of(stem)) as f:
        rec = json.load(f)
    rec["pred"] = np.array([float(v) for v in rec["pred"]], dtype=np.float64)
    return rec


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("names", nargs="*", help="file stems to (re)write; default all")
    ap.add_argument("--procs", type=int, default=min(8, os.cpu_count() or 1))
    args = ap.parse_args()
    for stem, w, rnd in BATCHES:
        if args.names and stem not in args.names:
            continue
        print(f"{stem}: oracle over the whole batch with {args.procs} processes", flush=True)
        rec = compute(stem, w, rnd, args.procs)
        with open(path_of(stem), "w") as f:
            json.dump(rec, f, indent=0)
            f.write("\n")
        print(f"{stem}: wrote {path_of(stem)} ({rec['oracle_seconds']} s)", flush=True)


if __name__ == "__main__":
    main()
