"""Pins of the sort-based ISRTF select oracle.

* the hand-computed two-request example built on the paper's iterative
  prediction example (tests/golden/srtf_two_requests.json);
* numpy.lexsort, an independent library sort, on random and adversarial inputs;
* closed-form special cases: all-equal predictions reduce to FCFS, k >= n is a
  full sort, k = 0 is empty, the cut separates the chosen from the rest.
"""
import json
import os

import numpy as np
import pytest

from oracle import oracle_order, oracle_select

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "srtf_two_requests.json")


def test_worked_example_golden():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        got = oracle_select(np.array(c["pred"], np.float32), np.array(c["arrival_seq"], np.int64),
                            c["batch_cap"])
        assert got.tolist() == c["selected"], c["what"]


def _lexsort_ref(pred, arr, k):
    # numpy.lexsort sorts NaN last and treats -0 == +0 when comparing floats;
    # map every NaN to one value so that NaNs tie with each other.
    p = np.where(np.isnan(pred), np.float32(np.nan), pred).astype(np.float64)
    nan = np.isnan(p)
    p = np.where(nan, 0.0, p)
    order = np.lexsort((np.arange(len(p)), arr, p, nan))
    return order[:min(k, len(p))]


SPECIALS = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, 1e-45, -1e-45, 1e-40,
                     3.4e38, -3.4e38, 1.0, 1.0, 2.5], dtype=np.float32)


@pytest.mark.parametrize("seed", range(12))
def test_matches_lexsort(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    kind = seed % 3
    if kind == 0:
        pred = rng.standard_normal(n).astype(np.float32) * 100
    elif kind == 1:
        pred = rng.integers(0, 5, size=n).astype(np.float32)  # many ties
    else:
        pred = rng.choice(SPECIALS, size=n)
    arr = rng.integers(0, max(2, n // 3), size=n).astype(np.int64)  # repeated arrivals too
    for k in (0, 1, n // 2, n, n + 7):
        got = oracle_select(pred, arr, k)
        assert got.tolist() == _lexsort_ref(pred, arr, k).tolist()


def test_all_equal_reduces_to_fcfs():
    arr = np.array([7, 3, 9, 1, 4], dtype=np.int64)
    pred = np.full(5, 42.0, np.float32)
    assert oracle_select(pred, arr, 3).tolist() == [3, 1, 4]


def test_full_sort_and_empty():
    pred = np.array([3.0, 1.0, 2.0], np.float32)
    arr = np.zeros(3, np.int64)
    assert oracle_select(pred, arr, 10).tolist() == [1, 2, 0]
    assert oracle_select(pred, arr, 0).tolist() == []


def test_signed_zero_and_nan_order():
    pred = np.array([np.nan, 0.0, -0.0, np.inf, -np.nan], np.float32)
    arr = np.array([0, 2, 1, 3, 4], np.int64)
    # -0 == +0: tie broken by arrival (index 2 arrived before index 1); NaNs after +inf
    assert oracle_order(pred, arr) == [2, 1, 3, 0, 4]


@pytest.mark.parametrize("seed", range(5))
def test_cut_property(seed):
    rng = np.random.default_rng(100 + seed)
    pred = rng.standard_normal(200).astype(np.float32)
    arr = rng.permutation(200).astype(np.int64)
    sel = set(oracle_select(pred, arr, 50).tolist())
    worst_in = max((pred[i], arr[i]) for i in sel)
    best_out = min((pred[i], arr[i]) for i in range(200) if i not in sel)
    assert worst_in < best_out
