"""Host logic of the round driver: the predictor input of a job."""
import numpy as np

import oracle
from paper_2505_09142_amd.driver import build_input


def test_build_input_matches_oracle_definition():
    rng = np.random.default_rng(0)
    for _ in range(3000):
        p = rng.integers(1, 50, size=int(rng.integers(1, 20))).astype(np.int32)
        r = rng.integers(50, 99, size=int(rng.integers(1, 30))).astype(np.int32)
        g = int(rng.integers(0, len(r) + 1))
        mp = int(rng.integers(2, 40))
        assert np.array_equal(build_input(p, r, g, mp), oracle.job_input(p, r, g, mp))


def test_build_input_examples():
    p = np.array([7, 8, 9], np.int32)
    r = np.array([1, 2, 3, 4], np.int32)
    assert build_input(p, r, 0, 10).tolist() == [7, 8, 9]
    assert build_input(p, r, 2, 10).tolist() == [7, 8, 9, 1, 2]
    assert build_input(p, r, 4, 4).tolist() == [7, 2, 3, 4]
    assert build_input(p, r, 4, 6).tolist() == [7, 9, 1, 2, 3, 4]
