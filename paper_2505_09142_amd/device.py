"""Device-side plumbing around libelis: weights resident in HBM, workspaces, streams.

PyTorch is used here only to own device memory and to name the current HIP
stream; every step of the predictor and of the selection runs in libelis'
kernels, reached through the same-named calls of ``_elis``.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _elis as E

BF16_KEYS = ("word", "pos", "w_qkv", "w_o", "w_1", "w_2")


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _to_dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device)  # bf16 bit patterns
    if a.dtype == np.float32:
        return torch.from_numpy(a).to(device)
    raise TypeError(a.dtype)


def config_of(shape) -> E.elis_config:
    """elis_config from any object with the encoder-shape attributes."""
    return E.elis_config(shape.n_layers, shape.d_model, shape.n_heads, shape.d_ff, shape.vocab, shape.max_pos,
                         shape.pooling, shape.head_hidden, shape.n_head_layers, shape.head_act, shape.ln_eps,
                         shape.out_scale, shape.out_shift)


class DeviceWeights:
    """Uploads one predictor's parameters and builds the elis_weights struct.

    ``tensors`` is a dict in the layout of include/elis.h: bf16 bit patterns
    (uint16) for the embedding tables and the four layer matrices, fp32 for the
    rest; per-layer entries are lists.
    """

    def __init__(self, shape, tensors: dict, device="cuda"):
        self.shape = shape
        self.cfg = config_of(shape)
        self.t = {}
        for k, v in tensors.items():
            self.t[k] = [_to_dev(x, device) for x in v] if isinstance(v, list) else _to_dev(v, device)
        L = shape.n_layers
        self._layers = (E.elis_layer_weights * max(1, L))()
        for l in range(L):
            y = self._layers[l]
            for name in ("w_qkv", "w_o", "w_1", "w_2", "b_qkv", "b_o", "b_1", "b_2", "ln1_g", "ln1_b", "ln2_g",
                         "ln2_b"):
                setattr(y, name, self.t[name][l].data_ptr())
        p = lambda k: self.t[k].data_ptr() if k in self.t else None
        nmid = len(self.t.get("head_mid_w", []))
        self._mid_w = (ctypes.c_void_p * max(1, nmid))(*[x.data_ptr() for x in self.t.get("head_mid_w", [])])
        self._mid_b = (ctypes.c_void_p * max(1, nmid))(*[x.data_ptr() for x in self.t.get("head_mid_b", [])])
        mid = lambda a: ctypes.cast(a, ctypes.POINTER(ctypes.c_void_p)) if nmid else None
        self.struct = E.elis_weights(self.cfg, p("word"), p("pos"), p("type0"), p("emb_ln_g"), p("emb_ln_b"),
                                     ctypes.cast(self._layers, ctypes.POINTER(E.elis_layer_weights)),
                                     p("head_w1"), p("head_b1"), p("head_w2"), p("head_b2"),
                                     mid(self._mid_w), mid(self._mid_b))


class Workspace:
    """A growable, 256-byte-aligned device scratch buffer owned by torch."""

    def __init__(self, device="cuda"):
        self.device = device
        self.buf = None

    def get(self, nbytes: int) -> tuple[int, int]:
        nbytes = max(256, int(nbytes))
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.buf.data_ptr()
        aligned = (base + 255) // 256 * 256
        return aligned, self.buf.numel() - (aligned - base)


class Predictor:
    """elis_predict_remaining + elis_isrtf_select on resident weights."""

    def __init__(self, weights: DeviceWeights, device="cuda"):
        self.w = weights
        self.device = device
        self.ws = Workspace(device)
        self.sel_ws = Workspace(device)

    def predict(self, token_ids: torch.Tensor, cu_seqlens: torch.Tensor, max_seqlen: int, out_pred=None,
                want_hidden=False, stream=None):
        n = cu_seqlens.numel() - 1
        T = token_ids.numel()
        need = E.elis_predict_workspace_bytes(self.w.cfg, T, n, max_seqlen)
        if need == 0:
            raise E.ElisError(E.ELIS_EINVAL, "elis_predict_workspace_bytes")
        ws, wsb = self.ws.get(need)
        if out_pred is None:
            out_pred = torch.empty(n, dtype=torch.float32, device=self.device)
        hid = torch.empty((T, self.w.shape.d_model), dtype=torch.float32, device=self.device) if want_hidden else None
        st = E.elis_predict_remaining(self.w.struct, token_ids.data_ptr(), cu_seqlens.data_ptr(), n, T, max_seqlen,
                                      out_pred.data_ptr(), hid.data_ptr() if hid is not None else None, ws, wsb,
                                      _stream(stream))
        E.check(st, "elis_predict_remaining")
        return out_pred, hid

    def status(self, stream=None):
        ws, _ = self.ws.get(0)
        return E.elis_read_status(ws, _stream(stream))

    def select(self, pred: torch.Tensor, arrival: torch.Tensor, batch_cap: int, out_idx=None, out_count=None,
               stream=None):
        n = pred.numel()
        if out_idx is None:
            out_idx = torch.full((max(1, batch_cap),), -1, dtype=torch.int32, device=self.device)
        if out_count is None:
            out_count = torch.zeros(1, dtype=torch.int32, device=self.device)
        ws, wsb = self.sel_ws.get(E.elis_select_workspace_bytes(n))
        st = E.elis_isrtf_select(pred.data_ptr(), arrival.data_ptr(), n, batch_cap, out_idx.data_ptr(),
                                 out_count.data_ptr(), ws, wsb, _stream(stream))
        E.check(st, "elis_isrtf_select")
        return out_idx, out_count


def upload_batch(batch, device="cuda"):
    """(token_ids, cu_seqlens, arrival_seq) of a packed batch as device tensors."""
    return (torch.from_numpy(batch.token_ids).to(device), torch.from_numpy(batch.cu_seqlens).to(device),
            torch.from_numpy(batch.arrival_seq).to(device))


class JobTable:
    """Device-resident job table (elis_jobs_*): per job slot the first token, a ring of the most
    recent max_pos - 1 tokens, the length, the cached prediction and the arrival number."""

    def __init__(self, max_jobs: int, max_pos: int, device="cuda", stream=None):
        nbytes = E.elis_jobs_table_bytes(max_jobs, max_pos)
        if nbytes == 0:
            raise E.ElisError(E.ELIS_EINVAL, "elis_jobs_table_bytes")
        self.device = device
        self.buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        base = (self.buf.data_ptr() + 255) // 256 * 256
        self.t = E.elis_job_table(base, max_jobs, max_pos)
        self.max_jobs, self.max_pos = max_jobs, max_pos
        self.sel_ws = Workspace(device)
        E.check(E.elis_jobs_init(self.t, _stream(stream)), "elis_jobs_init")

    def start(self, slots: torch.Tensor, arrival: torch.Tensor, stream=None):
        E.check(E.elis_jobs_start(self.t, slots.data_ptr(), arrival.data_ptr(), slots.numel(), _stream(stream)),
                "elis_jobs_start")

    def append(self, slots: torch.Tensor, offsets: torch.Tensor, tokens: torch.Tensor, total: int, stream=None):
        E.check(E.elis_jobs_append(self.t, slots.data_ptr(), offsets.data_ptr(),
                                   tokens.data_ptr() if total > 0 else None, slots.numel(), total, _stream(stream)),
                "elis_jobs_append")

    def pack(self, slots: torch.Tensor, total: int, max_seqlen: int, out_ids: torch.Tensor, out_cu: torch.Tensor,
             stream=None):
        E.check(E.elis_jobs_pack(self.t, slots.data_ptr(), slots.numel(), total, max_seqlen, out_ids.data_ptr(),
                                 out_cu.data_ptr(), _stream(stream)), "elis_jobs_pack")

    def store_pred(self, slots: torch.Tensor, pred: torch.Tensor, stream=None):
        E.check(E.elis_jobs_store_pred(self.t, slots.data_ptr(), pred.data_ptr(), slots.numel(), _stream(stream)),
                "elis_jobs_store_pred")

    def select(self, slots: torch.Tensor, batch_cap: int, out_slots: torch.Tensor, out_count: torch.Tensor,
               stream=None, wait: torch.Tensor | None = None, aging: float = 0.0):
        """Select over the cached keys; with `wait` (fp32 seconds per candidate) the keys are aged by
        `aging` tokens per second (elis_jobs_select_aged)."""
        a = slots.numel()
        ws, wsb = self.sel_ws.get(E.elis_jobs_select_workspace_bytes(a))
        if wait is None:
            E.check(E.elis_jobs_select(self.t, slots.data_ptr(), a, batch_cap, out_slots.data_ptr(),
                                       out_count.data_ptr(), ws, wsb, _stream(stream)), "elis_jobs_select")
        else:
            E.check(E.elis_jobs_select_aged(self.t, slots.data_ptr(), wait.data_ptr(), aging, a, batch_cap,
                                            out_slots.data_ptr(), out_count.data_ptr(), ws, wsb, _stream(stream)),
                    "elis_jobs_select_aged")

    def status(self, stream=None):
        return E.elis_read_status(self.t.base, _stream(stream))
