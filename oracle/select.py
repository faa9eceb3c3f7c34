"""Sort-based oracle of the ISRTF batch selection.

TEST INFRASTRUCTURE ONLY (imported by tests, the smoke check and the
benchmark's CPU-baseline leg; never by the product path).

ISRTF gives the highest priority to the job with the fewest predicted
remaining tokens and forms the batch starting from the highest priority
(Sec. 4.1, the Batcher of Alg. 1). Ties are broken by arrival order, i.e. the
FCFS order of the paper's baseline (Sec. 6.1), and then by index so that the
order is total. Reading of floating-point corner cases: -0 equals +0, and NaN
(any payload) ranks after +inf, all NaNs equal to each other.
"""
from __future__ import annotations

import math

import numpy as np


def _rank_key(i: int, pred, arrival):
    p = float(pred[i])
    if math.isnan(p):
        return (1, 0.0, int(arrival[i]), i)
    return (0, p, int(arrival[i]), i)


def oracle_order(pred, arrival_seq) -> list:
    """All indices, highest priority first."""
    n = len(pred)
    return sorted(range(n), key=lambda i: _rank_key(i, pred, arrival_seq))


def oracle_select(pred, arrival_seq, batch_cap: int) -> np.ndarray:
    """The first min(batch_cap, n) indices of the priority order, as int32."""
    order = oracle_order(pred, arrival_seq)
    return np.asarray(order[:max(0, min(batch_cap, len(order)))], dtype=np.int32)
