"""Scheduling-round driver: builds the predictor input of the jobs to re-score,
moves it to the device, and runs elis_predict_remaining then elis_isrtf_select.

The predictor input of a job is its prompt followed by the tokens it has
generated so far (Sec. 3.3; Predictor.iter of Alg. 1). When that is longer
than the encoder's position table, the first token (the CLS slot) is kept
together with the most recent max_pos - 1 tokens, so new tokens keep reaching
the predictor.
"""
from __future__ import annotations

import numpy as np
import torch

from .device import JobTable, Predictor


def build_input(prompt: np.ndarray, response: np.ndarray, generated: int, max_pos: int) -> np.ndarray:
    n_p = len(prompt)
    total = n_p + generated
    if total <= max_pos:
        out = np.empty(total, dtype=np.int32)
        out[:n_p] = prompt
        out[n_p:] = response[:generated]
        return out
    out = np.empty(max_pos, dtype=np.int32)
    out[0] = prompt[0] if n_p else response[0]
    tail_start = total - (max_pos - 1)          # index into prompt ‖ response
    k = 1
    if tail_start < n_p:
        seg = prompt[tail_start:]
        out[k:k + len(seg)] = seg
        k += len(seg)
        out[k:] = response[:generated]
    else:
        out[k:] = response[tail_start - n_p:generated]
    return out


class RoundDriver:
    """Packs a re-score set and runs predict + select on one stream.

    Host staging buffers are pinned and grow on demand; device buffers are
    torch allocations reused across rounds.
    """

    def __init__(self, predictor: Predictor, max_pos: int, device="cuda"):
        self.pr = predictor
        self.max_pos = max_pos
        self.device = device
        self._h_ids = torch.empty(0, dtype=torch.int32).pin_memory()
        self._h_cu = torch.empty(0, dtype=torch.int32).pin_memory()
        self._d_ids = torch.empty(0, dtype=torch.int32, device=device)
        self._d_cu = torch.empty(0, dtype=torch.int32, device=device)
        self._copied = None  # event recorded after the last host-to-device copy

    def _ensure(self, T: int, n: int):
        if self._h_ids.numel() < T:
            cap = max(T, 2 * self._h_ids.numel())
            self._h_ids = torch.empty(cap, dtype=torch.int32).pin_memory()
            self._d_ids = torch.empty(cap, dtype=torch.int32, device=self.device)
        if self._h_cu.numel() < n + 1:
            cap = max(n + 1, 2 * self._h_cu.numel())
            self._h_cu = torch.empty(cap, dtype=torch.int32).pin_memory()
            self._d_cu = torch.empty(cap, dtype=torch.int32, device=self.device)

    def pack(self, inputs: list) -> tuple[int, int, int]:
        """Writes the inputs back to back into the pinned staging buffers; returns (n, T, max_len)."""
        if self._copied is not None:
            self._copied.synchronize()  # the staging buffers are still being read by the last copy
        n = len(inputs)
        lens = np.fromiter((len(x) for x in inputs), dtype=np.int64, count=n)
        T = int(lens.sum())
        self._ensure(T, n)
        cu = self._h_cu.numpy()
        cu[0] = 0
        cu[1:n + 1] = np.cumsum(lens)
        ids = self._h_ids.numpy()
        for i, x in enumerate(inputs):
            ids[cu[i]:cu[i + 1]] = x
        return n, T, int(lens.max())

    def upload(self, n: int, T: int):
        self._d_ids[:T].copy_(self._h_ids[:T], non_blocking=True)
        self._d_cu[:n + 1].copy_(self._h_cu[:n + 1], non_blocking=True)
        self._copied = torch.cuda.Event()
        self._copied.record()
        return self._d_ids[:T], self._d_cu[:n + 1]

    def predict_inputs(self, inputs: list, out_pred: torch.Tensor | None = None) -> torch.Tensor:
        n, T, mx = self.pack(inputs)
        ids, cu = self.upload(n, T)
        pred, _ = self.pr.predict(ids, cu, mx, out_pred=out_pred)
        return pred

    def predict_jobs(self, job_ids, prompts, responses, generated) -> np.ndarray:
        inputs = [build_input(prompts[j], responses[j], int(generated[j]), self.max_pos) for j in job_ids]
        pred = self.predict_inputs(inputs)
        return pred.cpu().numpy()

    def select(self, pred: np.ndarray | torch.Tensor, arrival: np.ndarray, batch_cap: int) -> np.ndarray:
        d_pred = pred if isinstance(pred, torch.Tensor) else torch.from_numpy(
            np.ascontiguousarray(pred, dtype=np.float32)).to(self.device)
        d_arr = torch.from_numpy(np.ascontiguousarray(arrival, dtype=np.int64)).to(self.device)
        idx, cnt = self.pr.select(d_pred, d_arr, batch_cap)
        m = int(cnt.item())
        return idx[:m].cpu().numpy()


class DeviceRoundDriver:
    """Scheduling rounds on the device-resident job table.

    A job holds a table slot from start() to release(). The host keeps only integer
    bookkeeping (slots, tokens appended per job) to size launches; token contents stay
    in HBM. A round appends the tokens each job gained since its last append (the prompt
    when it starts), packs the re-score set on the device, predicts, caches the
    predictions in the table, and selects over the cached predictions of the
    candidates; the chosen slots are the round's only device-to-host transfer.
    Every upload of a call goes through one pinned staging buffer in one copy.
    """

    def __init__(self, predictor: Predictor, max_jobs: int, max_pos: int, device="cuda"):
        self.pr = predictor
        self.max_jobs, self.max_pos = max_jobs, max_pos
        self.device = device
        self.table = JobTable(max_jobs, max_pos, device)
        self.appended = {}                     # job -> tokens appended so far (prompt + generated)
        self.slot_of = {}                      # job -> table slot
        self.job_of = np.full(max_jobs, -1, dtype=np.int64)
        self.free = list(range(max_jobs - 1, -1, -1))
        self._h = torch.empty(1 << 16, dtype=torch.int32).pin_memory()
        self._d = torch.empty(1 << 16, dtype=torch.int32, device=device)
        self._ids = torch.empty(0, dtype=torch.int32, device=device)
        self._cu = torch.empty(0, dtype=torch.int32, device=device)
        self._out_slots = torch.empty(0, dtype=torch.int32, device=device)
        self._out_count = torch.zeros(1, dtype=torch.int32, device=device)
        self._copied = None
        self.h2d_bytes = 0  # host-to-device bytes uploaded so far
        self.d2h_bytes = 0

    def slot(self, job: int) -> int:
        return self.slot_of[job]

    def _upload(self, *parts):
        """Concatenates int32 / int64 arrays into the pinned staging buffer, copies it to the
        device in one transfer, and returns device views of the parts (int64 parts viewed
        back as int64)."""
        words = [np.ascontiguousarray(p).view(np.int32) if p.dtype in (np.int64, np.float32) else
                 np.ascontiguousarray(p, dtype=np.int32) for p in parts]
        # int64 parts start on an even word so the view back is 8-byte aligned
        offs, n = [], 0
        for w, p in zip(words, parts):
            n += n & 1 if p.dtype == np.int64 else 0
            offs.append(n)
            n += len(w)
        if self._copied is not None:
            self._copied.synchronize()  # the last copy may still read the staging buffer
        if self._h.numel() < n:
            cap = max(n, 2 * self._h.numel())
            self._h = torch.empty(cap, dtype=torch.int32).pin_memory()
            self._d = torch.empty(cap, dtype=torch.int32, device=self.device)
        h = self._h.numpy()
        for o, w in zip(offs, words):
            h[o:o + len(w)] = w
        # The device buffer is reused by the next upload: stream order keeps the kernels
        # that read this one ahead of that copy.
        self._d[:n].copy_(self._h[:n], non_blocking=True)
        self.h2d_bytes += 4 * n
        self._copied = torch.cuda.Event()
        self._copied.record()
        out = []
        for o, w, p in zip(offs, words, parts):
            v = self._d[o:o + len(w)]
            out.append(v.view(torch.int64) if p.dtype == np.int64 else
                       v.view(torch.float32) if p.dtype == np.float32 else v)
        return out

    def release(self, jobs):
        """Jobs that finished give their slots back."""
        for j in jobs:
            s = self.slot_of.pop(j)
            self.job_of[s] = -1
            self.free.append(s)
            del self.appended[j]

    def start(self, jobs, arrival_seq):
        """Empty slots for new jobs with their arrival numbers."""
        if len(jobs) == 0:
            return
        if len(jobs) > len(self.free):
            raise RuntimeError(f"job table full ({self.max_jobs} slots)")
        for j in jobs:
            s = self.free.pop()
            self.slot_of[j] = s
            self.job_of[s] = j
            self.appended[j] = 0
        slots = np.array([self.slot_of[j] for j in jobs], dtype=np.int32)
        d_slots, d_arr = self._upload(slots, np.asarray(arrival_seq, dtype=np.int64))
        self.table.start(d_slots, d_arr)

    def sync_tokens(self, jobs, prompts, responses, generated):
        """Appends to each job the tokens it gained since its last append: the prompt when it
        starts, then responses[j][:generated[j]]; only that new tail crosses to the device."""
        slots, offs, toks = [], [0], []
        for j in jobs:
            n_p, done = len(prompts[j]), self.appended[j]
            g = int(generated[j])
            if n_p + g <= done:
                continue
            if done < n_p:
                toks.append(prompts[j][done:])
                toks.append(responses[j][:g])
            else:
                toks.append(responses[j][done - n_p:g])
            new = (n_p + g) - done
            slots.append(self.slot_of[j])
            offs.append(offs[-1] + new)
            self.appended[j] = n_p + g
        if not slots:
            return
        d_slots, d_off, d_tok = self._upload(np.array(slots, dtype=np.int32), np.array(offs, dtype=np.int32),
                                             np.concatenate(toks))
        self.table.append(d_slots, d_off, d_tok, offs[-1])

    def predict(self, jobs, out_pred: torch.Tensor | None = None) -> torch.Tensor:
        """Packs the jobs' inputs on the device, predicts, caches the predictions in the table;
        returns them as a device tensor (no synchronisation)."""
        lens = np.fromiter((min(self.appended[j], self.max_pos) for j in jobs), dtype=np.int64, count=len(jobs))
        T, n, mx = int(lens.sum()), len(jobs), int(lens.max())
        if self._ids.numel() < T:
            self._ids = torch.empty(max(T, 2 * self._ids.numel()), dtype=torch.int32, device=self.device)
        if self._cu.numel() < n + 1:
            self._cu = torch.empty(max(n + 1, 2 * self._cu.numel()), dtype=torch.int32, device=self.device)
        (d_slots,) = self._upload(np.fromiter((self.slot_of[j] for j in jobs), dtype=np.int32, count=n))
        ids, cu = self._ids[:T], self._cu[:n + 1]
        self.table.pack(d_slots, T, mx, ids, cu)
        pred, _ = self.pr.predict(ids, cu, mx, out_pred=out_pred)
        self.table.store_pred(d_slots, pred)
        return pred

    def store_keys(self, jobs, keys) -> None:
        """Caches priority keys computed outside the encoder (FCFS, SJF, a stand-in predictor)."""
        d_slots, d_keys = self._upload(np.fromiter((self.slot_of[j] for j in jobs), dtype=np.int32, count=len(jobs)),
                                       np.asarray(keys, dtype=np.float32))
        self.table.store_pred(d_slots, d_keys)

    def select(self, candidates, batch_cap: int, wait=None, aging: float = 0.0) -> np.ndarray:
        """Chosen job ids among the candidates (cached keys, ties by arrival number); with `wait`
        (fp32 seconds per candidate) the keys are aged on the device by `aging` per second."""
        n = len(candidates)
        slots = np.fromiter((self.slot_of[j] for j in candidates), dtype=np.int32, count=n)
        if wait is None:
            (d_slots,) = self._upload(slots)
            d_wait = None
        else:
            d_slots, d_wait = self._upload(slots, np.asarray(wait, dtype=np.float32))
        if self._out_slots.numel() < max(1, batch_cap):
            self._out_slots = torch.empty(max(1, batch_cap), dtype=torch.int32, device=self.device)
        self.table.select(d_slots, batch_cap, self._out_slots, self._out_count, wait=d_wait, aging=aging)
        # one transfer back: the count and the chosen slots
        res = torch.cat([self._out_count, self._out_slots[:min(batch_cap, n)]]).cpu().numpy()
        self.d2h_bytes += 4 * len(res)
        return self.job_of[res[1:1 + int(res[0])]]


class HostRoundDriver:
    """The same round interface as DeviceRoundDriver with host-side packing: every re-scored
    job's whole input is rebuilt on the host and copied to the device each round, and the
    candidates' predictions and arrival numbers are copied back in for the select."""

    def __init__(self, predictor: Predictor, max_pos: int, n_jobs: int, device="cuda"):
        self.rd = RoundDriver(predictor, max_pos, device)
        self.max_pos = max_pos
        self.pred = np.full(n_jobs, np.nan, dtype=np.float32)
        self.h2d_bytes = 0  # host-to-device bytes uploaded so far
        self.d2h_bytes = 0
        self._g = None
        self._p = None
        self._r = None

    def start(self, jobs, arrival_seq):
        pass

    def release(self, jobs):
        pass

    def sync_tokens(self, jobs, prompts, responses, generated):
        self._p, self._r, self._g = prompts, responses, generated

    def predict(self, jobs, out_pred=None):
        inputs = [build_input(self._p[j], self._r[j], int(self._g[j]), self.max_pos) for j in jobs]
        pred = self.rd.predict_inputs(inputs, out_pred=out_pred)
        self.pred[list(jobs)] = pred.cpu().numpy()
        self.h2d_bytes += 4 * (sum(len(x) for x in inputs) + len(inputs) + 1)
        self.d2h_bytes += 4 * len(inputs)
        return pred

    def store_keys(self, jobs, keys) -> None:
        self.pred[list(jobs)] = np.asarray(keys, dtype=np.float32)

    def select(self, candidates, batch_cap: int, wait=None, aging: float = 0.0) -> np.ndarray:
        if wait is not None:
            raise NotImplementedError("aged keys need the device job table (DeviceRoundDriver)")
        cand = np.asarray(candidates, dtype=np.int64)
        local = self.rd.select(self.pred[cand], cand, batch_cap)
        self.h2d_bytes += 12 * len(cand)
        self.d2h_bytes += 4 * (len(local) + 1)
        return cand[local]
