"""Collects the observed parity margins of a GPU test run.

Each full-size or end-to-end parity test records what it measured (largest
hidden-state error, largest prediction error, the oracle's gap at the batch
cut, ...). When the environment variable ELIS_PARITY_SUMMARY names a file, the
session writes those records there as a markdown table at the end of the run
(tests/conftest.py); the bars themselves are asserted by the tests.
"""
from __future__ import annotations

RECORDS: list = []


def record(case: str, **fields) -> None:
    RECORDS.append({"case": case, **fields})


def _fmt(v) -> str:
    if isinstance(v, bool):
        return "yes" if v else "no"
    if isinstance(v, float):
        return f"{v:.3e}"
    return str(v)


def write_summary(path: str, header: str) -> None:
    cols = []
    for r in RECORDS:
        for k in r:
            if k not in cols:
                cols.append(k)
    lines = [header, "", "| " + " | ".join(cols) + " |", "|" + "---|" * len(cols)]
    for r in RECORDS:
        lines.append("| " + " | ".join(_fmt(r.get(c, "")) for c in cols) + " |")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
