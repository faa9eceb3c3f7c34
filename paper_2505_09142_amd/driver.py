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

from .device import Predictor


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
