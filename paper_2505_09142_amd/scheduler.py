"""The scheduling loop of one node (Alg. 1) on a synthetic decode clock.

Each round: admit the requests that have arrived into the Job Pool; give the
Job-Pool jobs (new arrivals and the jobs that ran in the last window) a fresh
priority key while every other job keeps its cached key; form the batch from
the `batch_cap` candidates with the smallest keys, ties by arrival (Sec. 4.1;
a running job not chosen again is preempted); run one window: every chosen job
generates min(window, tokens it has left) tokens at `step_cost` seconds per
decode step, and the window lasts until every chosen job has done so (end_rule
"all") or until the first one has ("first").

Keys by policy:
  "isrtf"  predicted remaining tokens: the encoder on the device re-scores the
           prompt plus the generated tokens (Sec. 3.3), or, when `key_fn` is
           given, the keys it returns (a stand-in predictor of known accuracy);
  "fcfs"   0 for every job, so the arrival order decides (Sec. 6.1 baseline);
  "sjf"    the true total response length (the oracle baseline of Sec. 6.1).

Starvation control and preemption cost (Sec. 3.4 leaves both open):
  aging         a candidate that has waited w seconds since it last ran (or
                arrived) is ranked by key - aging * w, on the device
                (elis_jobs_select_aged);
  prefill_cost  a preempted job that is chosen again first re-prefills its
                prompt and generated tokens at prefill_cost seconds per token;
                the window waits for it.

The round driver (DeviceRoundDriver or HostRoundDriver) owns the predictor,
the key cache and the selection; the loop itself is host bookkeeping only.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field

import numpy as np

POLICIES = ("isrtf", "fcfs", "sjf")


@dataclass
class Round:
    t: float
    rescored: list
    pred: np.ndarray  # the re-scored jobs' new keys
    candidates: list
    chosen: list
    steps: int
    latency_s: float  # host wall time of key update + select (selection on the host)
    wait: np.ndarray = None   # fp32 seconds waited, aligned with candidates (aging only)
    resumed: list = None      # preempted jobs that re-prefilled this round
    prefill_s: float = 0.0


@dataclass
class ScheduleResult:
    rounds: list = field(default_factory=list)
    finish_t: np.ndarray = None
    jct: np.ndarray = None
    queue_delay: np.ndarray = None
    preemptions: np.ndarray = None
    generated: np.ndarray = None


def run_schedule(arrival_t, prompts, responses, driver, *, window: int, step_cost: float, batch_cap: int,
                 policy: str = "isrtf", key_fn=None, rescore: str = "pool", end_rule: str = "all",
                 max_rounds: int | None = None, aging: float = 0.0, prefill_cost: float = 0.0) -> ScheduleResult:
    if policy not in POLICIES:
        raise ValueError(policy)
    arrival_t = np.asarray(arrival_t, dtype=np.float64)
    n = len(arrival_t)
    total = np.array([len(r) for r in responses], dtype=np.int64)
    plen = np.array([len(p) for p in prompts], dtype=np.int64)
    gen = np.zeros(n, dtype=np.int64)
    finish = np.full(n, np.nan)
    ready = arrival_t.copy()
    preempted = np.zeros(n, dtype=np.int64)
    dropped = np.zeros(n, dtype=bool)   # KV cache dropped by a preemption, not yet re-prefilled
    running: set = set()
    job_pool: list = []
    last_batch: list = []
    next_arrival, finished, now = 0, 0, 0.0
    use_encoder = policy == "isrtf" and key_fn is None
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
        candidates = sorted(running)
        wait = None
        if aging != 0.0:
            wait = np.fromiter((now - ready[j] for j in candidates), dtype=np.float64,
                               count=len(candidates)).astype(np.float32)
        t0 = time.perf_counter()
        if not rescore_set:
            keys = np.zeros(0, dtype=np.float32)
        elif use_encoder:
            driver.sync_tokens(rescore_set, prompts, responses, gen)
            keys = driver.predict(rescore_set)  # stays on the device; read back after the loop
        else:
            if policy == "isrtf":
                keys = np.asarray(key_fn(rescore_set, gen), dtype=np.float32)
            elif policy == "sjf":
                keys = total[rescore_set].astype(np.float32)
            else:
                keys = np.zeros(len(rescore_set), dtype=np.float32)
            driver.store_keys(rescore_set, keys)
        chosen = [int(j) for j in driver.select(candidates, batch_cap, wait=wait, aging=aging)]
        latency = time.perf_counter() - t0
        in_batch = set(chosen)
        for j in last_batch:
            if j not in in_batch:
                dropped[j] = True
                preempted[j] += 1
        resumed = sorted(j for j in chosen if dropped[j])
        prefill_s = prefill_cost * sum(int(plen[j] + gen[j]) for j in resumed) if resumed else 0.0
        dropped[resumed] = False
        budget = {j: int(min(window, total[j] - gen[j])) for j in chosen}
        if end_rule == "all":
            steps = max(budget.values())
        elif end_rule == "first":
            steps = min(budget.values())
        else:
            raise ValueError(end_rule)
        end = now + prefill_s + steps * step_cost
        done_now = []
        last_batch = []
        for j in chosen:
            gained = min(budget[j], steps)
            gen[j] += gained
            if gen[j] == total[j]:
                finish[j] = now + prefill_s + gained * step_cost
                running.discard(j)
                finished += 1
                done_now.append(j)
            else:
                job_pool.append(j)
                last_batch.append(j)
                ready[j] = end
        driver.release(done_now)
        out.rounds.append(Round(now, rescore_set, keys, candidates, chosen, steps, latency, wait, resumed,
                                prefill_s))
        now = end
    for r in out.rounds:
        if not isinstance(r.pred, np.ndarray):
            r.pred = r.pred.cpu().numpy()
    out.finish_t = finish
    out.jct = finish - arrival_t
    out.queue_delay = out.jct - total * step_cost
    out.preemptions = preempted
    out.generated = gen
    return out


def run_isrtf(arrival_t, prompts, responses, driver, *, window: int, step_cost: float, batch_cap: int,
              rescore: str = "pool", end_rule: str = "all", max_rounds: int | None = None) -> ScheduleResult:
    """ISRTF with the encoder on the device re-scoring the Job Pool every round."""
    return run_schedule(arrival_t, prompts, responses, driver, window=window, step_cost=step_cost,
                        batch_cap=batch_cap, policy="isrtf", rescore=rescore, end_rule=end_rule,
                        max_rounds=max_rounds)
