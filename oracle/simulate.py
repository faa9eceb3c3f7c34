"""Oracle simulator of ELIS's scheduling flow on one node (Alg. 1, Sec. 4.1).

TEST INFRASTRUCTURE ONLY (imported by tests, the smoke check and the
benchmark's CPU-baseline leg; never by the product path).

Each iteration: the jobs in the Job Pool (new arrivals and jobs that ran in
the previous window) get a fresh priority key; every admitted, unfinished job
enters the priority buffer; the batcher takes the highest-priority jobs up to
the batch cap; the backend runs one window of K tokens (Sec. 4.1, backend
worker); finished jobs leave, the rest return to the Job Pool.

Priority keys (smaller runs first, ties by arrival order):
  * "isrtf": the predicted number of remaining tokens, re-predicted from the
    prompt plus the tokens generated so far (Sec. 3.3, Alg. 1);
  * "fcfs":  the same key for every job, so the arrival order decides
    (the baseline of Sec. 6.1);
  * "sjf":   the job's true total response length, known in advance (the
    oracle baseline of Sec. 6.1, which ranks by profiled length).

Starvation control and preemption cost (Sec. 3.4 says the system can tune
how often jobs are preempted but gives no algorithm; these are readings):
  * aging: a job that has waited w seconds since it last ran (or since its
    arrival) is ranked by key - aging * w; aging = 0 disables it. The aged key
    is evaluated in float64 from the float32 key, the float32 aging rate and
    the float32 wait, and rounded once to float32, the precision the select
    compares in;
  * prefill_cost: a job that ran, was left out of a later batch while
    unfinished (preempted: its KV cache is dropped) and is then chosen again
    must first re-prefill its prompt and generated tokens, prefill_cost
    seconds per token; the batch waits for it, so the window lasts
    prefill_cost * (re-prefilled tokens) + steps * step_cost.

Other readings of points the paper leaves open:
  * one backend worker, so no load balancing;
  * the LLM is replaced by a fixed cost per decode step of the batch, and the
    first prefill is free;
  * without prefill_cost a job that is not selected while it was running is
    preempted at no cost;
  * window end: every selected job stops after K tokens or at its end, and the
    window lasts until all have stopped ("all"); the alternative reading, the
    window ends at the first finish, is end_rule="first";
  * the predictor input is the prompt followed by the generated tokens; when
    longer than max_pos, the first token and the last max_pos - 1 tokens are
    kept;
  * queuing delay of a job = its JCT minus the decode time of its own tokens
    (R * step_cost): the time it spent waiting, including windows it was part
    of but had already stopped in, and re-prefills.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .select import oracle_select

POLICIES = ("isrtf", "fcfs", "sjf")


def job_input(prompt: np.ndarray, response: np.ndarray, g: int, max_pos: int) -> np.ndarray:
    """Predictor input of a job that has generated g tokens."""
    x = np.concatenate([np.asarray(prompt, dtype=np.int32), np.asarray(response[:g], dtype=np.int32)])
    if len(x) > max_pos:
        x = np.concatenate([x[:1], x[len(x) - (max_pos - 1):]])
    return x


def aged_keys(keys: np.ndarray, wait: np.ndarray, aging: float) -> np.ndarray:
    """float32(float64(key) - float64(aging) * float64(wait)) for float32 key, aging and wait."""
    k = np.asarray(keys, dtype=np.float32).astype(np.float64)
    w = np.asarray(wait, dtype=np.float32).astype(np.float64)
    a = np.float64(np.float32(aging))
    with np.errstate(over="ignore", invalid="ignore"):
        return (k - a * w).astype(np.float32)


@dataclass
class RoundRecord:
    t: float                 # simulated time at the start of the round
    rescored: list           # job ids given a new key this round (ascending)
    pred: np.ndarray         # their new keys (predictions for "isrtf"), aligned with rescored
    candidates: list         # admitted unfinished job ids (ascending)
    selected: list           # chosen job ids, highest priority first
    window_steps: int        # decode steps the window lasted
    keys: np.ndarray = None  # float32 keys the select ranked, aligned with candidates
    wait: np.ndarray = None  # float32 waits (seconds), aligned with candidates
    resumed: list = None     # preempted jobs that re-prefilled this round (ascending)
    prefill_s: float = 0.0   # re-prefill time at the start of the window


@dataclass
class SimResult:
    rounds: list = field(default_factory=list)
    finish_t: np.ndarray = None
    first_run_t: np.ndarray = None
    jct: np.ndarray = None
    queue_delay: np.ndarray = None
    preemptions: np.ndarray = None
    generated: np.ndarray = None


def simulate(arrival_t, prompts, responses, *, window: int, step_cost: float, batch_cap: int,
             max_pos: int, predict_fn=None, rescore: str = "pool", end_rule: str = "all",
             select_fn=None, max_rounds: int | None = None, policy: str = "isrtf",
             aging: float = 0.0, prefill_cost: float = 0.0) -> SimResult:
    """Run the scheduling loop until every job has finished (or max_rounds).

    arrival_t: non-decreasing arrival times; job id = arrival order.
    predict_fn(job_ids, inputs, g) -> predictions (one per job id); g is the
        per-job generated-token count array. Used by policy "isrtf" only.
    rescore: "pool" re-keys only Job-Pool jobs; "all" re-keys every admitted
        unfinished job each round.
    select_fn(keys, arrival_seq, batch_cap) -> indices; defaults to oracle_select.
    """
    if policy not in POLICIES:
        raise ValueError(policy)
    if policy == "isrtf" and predict_fn is None:
        raise ValueError("policy 'isrtf' needs predict_fn")
    sel_fn = oracle_select if select_fn is None else select_fn
    arrival_t = np.asarray(arrival_t, dtype=np.float64)
    N = len(arrival_t)
    R = np.array([len(r) for r in responses], dtype=np.int64)
    P = np.array([len(p) for p in prompts], dtype=np.int64)
    g = np.zeros(N, dtype=np.int64)
    key = np.full(N, np.nan, dtype=np.float32)
    ready_t = arrival_t.copy()          # when each job last became ready to run
    finish_t = np.full(N, np.nan)
    first_run_t = np.full(N, np.nan)
    preempt = np.zeros(N, dtype=np.int64)
    evicted = np.zeros(N, dtype=bool)   # preempted since it last ran: KV cache dropped
    active: set = set()
    pool: list = []
    ran_last: list = []                 # unfinished jobs of the previous window
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
        if todo and policy == "isrtf":
            inputs = [job_input(prompts[j], responses[j], int(g[j]), max_pos) for j in todo]
            p = np.asarray(predict_fn(todo, inputs, g), dtype=np.float64)
        elif todo and policy == "sjf":
            p = R[todo].astype(np.float64)
        elif todo:
            p = np.zeros(len(todo))
        else:
            p = np.zeros(0)
        key[todo] = p.astype(np.float32)
        cand = sorted(active)
        wait = np.asarray([t - ready_t[j] for j in cand], dtype=np.float64).astype(np.float32)
        k32 = key[cand] if aging == 0.0 else aged_keys(key[cand], wait, aging)
        local = sel_fn(k32, np.asarray(cand, dtype=np.int64), batch_cap)
        chosen = [cand[i] for i in local]
        chosen_set = set(chosen)
        for j in ran_last:
            if j not in chosen_set:
                evicted[j] = True
                preempt[j] += 1
        resumed = sorted(j for j in chosen if evicted[j])
        refill_tokens = sum(int(P[j] + g[j]) for j in resumed)
        prefill_s = prefill_cost * refill_tokens if resumed else 0.0
        for j in resumed:
            evicted[j] = False
        left = {j: int(min(window, R[j] - g[j])) for j in chosen}
        if end_rule == "all":
            steps = max(left.values())
        elif end_rule == "first":
            steps = min(left.values())
        else:
            raise ValueError(end_rule)
        end_t = t + prefill_s + steps * step_cost
        ran_last = []
        for j in chosen:
            if np.isnan(first_run_t[j]):
                first_run_t[j] = t
            gain = min(left[j], steps)
            g[j] += gain
            if g[j] == R[j]:
                finish_t[j] = t + prefill_s + gain * step_cost
                active.discard(j)
                done += 1
            else:
                pool.append(j)
                ran_last.append(j)
                ready_t[j] = end_t
        res.rounds.append(RoundRecord(t, todo, p, cand, chosen, steps, k32, wait, resumed, prefill_s))
        t = end_t
    res.finish_t = finish_t
    res.first_run_t = first_run_t
    res.jct = finish_t - arrival_t
    res.queue_delay = res.jct - R * step_cost
    res.preemptions = preempt
    res.generated = g
    return res
