"""The ISRTF scheduling loop of one node (Alg. 1) on a synthetic decode clock.

Each round: admit the requests that have arrived into the Job Pool; re-predict the
remaining length of the Job-Pool jobs only (new arrivals and the jobs that ran in
the last window; every other job keeps its cached prediction); form the batch from
the `batch_cap` candidates with the fewest predicted remaining tokens, ties by
arrival (Sec. 4.1; a running job not chosen again is preempted, at no cost here);
run one window: every chosen job generates min(window, tokens it has left) tokens
at `step_cost` seconds per decode step, and the window lasts until every chosen job
has done so (end_rule "all") or until the first one has ("first").

The round driver (DeviceRoundDriver or HostRoundDriver) owns the predictor and the
selection; the loop itself is host bookkeeping only.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Round:
    t: float
    rescored: list
    pred: np.ndarray  # the re-scored jobs' new predictions
    candidates: list
    chosen: list
    steps: int
    latency_s: float  # host wall time of sync + predict + select (selection on the host)


@dataclass
class ScheduleResult:
    rounds: list = field(default_factory=list)
    finish_t: np.ndarray = None
    jct: np.ndarray = None
    generated: np.ndarray = None


def run_isrtf(arrival_t, prompts, responses, driver, *, window: int, step_cost: float, batch_cap: int,
              rescore: str = "pool", end_rule: str = "all", max_rounds: int | None = None) -> ScheduleResult:
    arrival_t = np.asarray(arrival_t, dtype=np.float64)
    n = len(arrival_t)
    total = np.array([len(r) for r in responses], dtype=np.int64)
    gen = np.zeros(n, dtype=np.int64)
    finish = np.full(n, np.nan)
    running: set = set()
    job_pool: list = []
    next_arrival, finished, now = 0, 0, 0.0
    out = ScheduleResult()
    while finished < n and (max_rounds is None or len(out.rounds) < max_rounds):
        fresh = []
        while next_arrival < n and arrival_t[next_arrival] <= now:
            fresh.append(next_arrival)
            next_arrival += 1
        if fresh:
            driver.start(fresh, fresh)          # arrival number = arrival order
            running.update(fresh)
            job_pool.extend(fresh)
        if not running:
            now = float(arrival_t[next_arrival])
            continue
        rescore_set = sorted(job_pool) if rescore == "pool" else sorted(running)
        job_pool = []
        t0 = time.perf_counter()
        if rescore_set:
            driver.sync_tokens(rescore_set, prompts, responses, gen)
            pred = driver.predict(rescore_set)  # stays on the device; read back after the loop
        else:
            pred = np.zeros(0, dtype=np.float32)
        candidates = sorted(running)
        chosen = [int(j) for j in driver.select(candidates, batch_cap)]
        latency = time.perf_counter() - t0
        budget = {j: int(min(window, total[j] - gen[j])) for j in chosen}
        if end_rule == "all":
            steps = max(budget.values())
        elif end_rule == "first":
            steps = min(budget.values())
        else:
            raise ValueError(end_rule)
        done_now = []
        for j in chosen:
            gained = min(budget[j], steps)
            gen[j] += gained
            if gen[j] == total[j]:
                finish[j] = now + gained * step_cost
                running.discard(j)
                finished += 1
                done_now.append(j)
            else:
                job_pool.append(j)
        driver.release(done_now)
        out.rounds.append(Round(now, rescore_set, pred, candidates, chosen, steps, latency))
        now += steps * step_cost
    for r in out.rounds:
        if not isinstance(r.pred, np.ndarray):
            r.pred = r.pred.cpu().numpy()
    out.finish_t = finish
    out.jct = finish - arrival_t
    out.generated = gen
    return out
