"""Oracle simulator of ELIS's scheduling flow on one node (Alg. 1, Sec. 4.1).

TEST INFRASTRUCTURE ONLY (imported by tests, the smoke check and the
benchmark's CPU-baseline leg; never by the product path).

Each iteration: the jobs in the Job Pool (new arrivals and jobs that ran in
the previous window) get a fresh prediction of their remaining tokens from
their prompt plus what they have generated so far (Sec. 3.3, Alg. 1); every
admitted, unfinished job enters the priority buffer; the batcher takes the
highest-priority jobs up to the batch cap (ISRTF: fewest predicted remaining
tokens first); the backend runs one window of K tokens (Sec. 4.1, backend
worker); finished jobs leave, the rest return to the Job Pool.

Readings of points the paper leaves open:
  * one backend worker, so no load balancing;
  * the LLM is replaced by a fixed cost per decode step of the batch, and
    prefill is free;
  * a job that is not selected while it was running is preempted at no cost;
  * window end: every selected job stops after K tokens or at its end, and the
    window lasts until all have stopped ("all"); the alternative reading, the
    window ends at the first finish, is end_rule="first";
  * the predictor input is the prompt followed by the generated tokens; when
    longer than max_pos, the first token and the last max_pos - 1 tokens are
    kept.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .select import oracle_select


def job_input(prompt: np.ndarray, response: np.ndarray, g: int, max_pos: int) -> np.ndarray:
    """Predictor input of a job that has generated g tokens."""
    x = np.concatenate([np.asarray(prompt, dtype=np.int32), np.asarray(response[:g], dtype=np.int32)])
    if len(x) > max_pos:
        x = np.concatenate([x[:1], x[len(x) - (max_pos - 1):]])
    return x


@dataclass
class RoundRecord:
    t: float                 # simulated time at the start of the round
    rescored: list           # job ids given a new prediction this round (ascending)
    pred: np.ndarray         # the new predictions, aligned with rescored
    candidates: list         # admitted unfinished job ids (ascending)
    selected: list           # chosen job ids, highest priority first
    window_steps: int        # decode steps the window lasted


@dataclass
class SimResult:
    rounds: list = field(default_factory=list)
    finish_t: np.ndarray = None
    first_run_t: np.ndarray = None
    jct: np.ndarray = None
    generated: np.ndarray = None


def simulate(arrival_t, prompts, responses, *, window: int, step_cost: float, batch_cap: int,
             max_pos: int, predict_fn, rescore: str = "pool", end_rule: str = "all",
             select_fn=None, max_rounds: int | None = None) -> SimResult:
    """Run the ISRTF loop until every job has finished (or max_rounds).

    arrival_t: non-decreasing arrival times; job id = arrival order.
    predict_fn(job_ids, inputs, g) -> predictions (one per job id); g is the
        per-job generated-token count array (for predictors that use it).
    rescore: "pool" re-predicts only Job-Pool jobs; "all" re-predicts every
        admitted unfinished job each round.
    select_fn(pred, arrival_seq, batch_cap) -> indices; defaults to oracle_select.
    """
    sel_fn = oracle_select if select_fn is None else select_fn
    arrival_t = np.asarray(arrival_t, dtype=np.float64)
    N = len(arrival_t)
    R = np.array([len(r) for r in responses], dtype=np.int64)
    g = np.zeros(N, dtype=np.int64)
    pred = np.full(N, np.nan, dtype=np.float64)
    finish_t = np.full(N, np.nan)
    first_run_t = np.full(N, np.nan)
    active: set = set()
    pool: list = []
    nxt = 0
    t = 0.0
    done = 0
    res = SimResult()
    while done < N:
        if max_rounds is not None and len(res.rounds) >= max_rounds:
            break
        while nxt < N and arrival_t[nxt] <= t:
            active.add(nxt)
            pool.append(nxt)
            nxt += 1
        if not active:
            t = float(arrival_t[nxt])
            continue
        todo = sorted(pool) if rescore == "pool" else sorted(active)
        pool = []
        if todo:
            inputs = [job_input(prompts[j], responses[j], int(g[j]), max_pos) for j in todo]
            p = np.asarray(predict_fn(todo, inputs, g), dtype=np.float64)
            pred[todo] = p
        else:
            p = np.zeros(0)
        cand = sorted(active)
        local = sel_fn(pred[cand].astype(np.float32), np.asarray(cand, dtype=np.int64), batch_cap)
        chosen = [cand[i] for i in local]
        left = {j: int(min(window, R[j] - g[j])) for j in chosen}
        if end_rule == "all":
            steps = max(left.values())
        elif end_rule == "first":
            steps = min(left.values())
        else:
            raise ValueError(end_rule)
        for j in chosen:
            if np.isnan(first_run_t[j]):
                first_run_t[j] = t
            gain = min(left[j], steps)
            g[j] += gain
            if g[j] == R[j]:
                finish_t[j] = t + gain * step_cost
                active.discard(j)
                done += 1
            else:
                pool.append(j)
        res.rounds.append(RoundRecord(t, todo, p, cand, chosen, steps))
        t += steps * step_cost
    res.finish_t = finish_t
    res.first_run_t = first_run_t
    res.jct = finish_t - arrival_t
    res.generated = g
    return res
