import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


@pytest.fixture(scope="session")
def repo_root():
    return ROOT


def pytest_sessionfinish(session, exitstatus):
    path = os.environ.get("ELIS_PARITY_SUMMARY")
    if not path:
        return
    from tests import parity_log
    if not parity_log.RECORDS:
        return
    cmd = os.environ.get("ELIS_PARITY_COMMAND", "python -m pytest -m gpu")
    header = ("# Observed parity margins (written by the GPU test run)\n\n"
              f"Command: `{cmd}` (exit status {int(exitstatus)}). One row per recorded check; "
              "hidden = max-abs over the compared rows (bar 5e-2), pred rel = max |p - p_ref| / max(|p_ref|, 1) "
              "(bar 2e-2), y rel = max |y - y_ref| / max |y_ref| for the unshifted head output y = "
              "(p - out_shift) / out_scale (bar 2e-2), gap = the oracle's key gap at the batch cut, "
              "margin ok = gap > 2 x max |p - p_ref| (then the selected sets must be equal).")
    parity_log.write_summary(path, header)
