"""ctypes binding of libelis (include/elis.h): argument marshalling only.

Every function below has the name of the C entry point it calls and passes
its arguments through unchanged (device pointers as Python ints, the stream
as a hipStream_t handle). All computation happens in the HIP kernels of
libelis.so; if the library is missing this module raises at import-use time,
and there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int, c_int32, c_size_t, c_uint32, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libelis.so")

ELIS_OK = 0
ELIS_EINVAL = -1
ELIS_ESHAPE = -2
ELIS_EWORKSPACE = -3
ELIS_EHIP = -4
ELIS_EDEVICE = -5
ELIS_EUNSUPPORTED = -6

ELIS_DEV_BAD_TOKEN = 1
ELIS_DEV_BAD_CU = 2
ELIS_DEV_LONG_SEQ = 4
ELIS_DEV_BAD_SLOT = 8
ELIS_DEV_PACK_SIZE = 16

ELIS_POOL_CLS = 0
ELIS_POOL_MEAN = 1

ELIS_ACT_RELU = 0
ELIS_ACT_IDENTITY = 1
ELIS_EPI_BIAS_BF16 = 0
ELIS_EPI_BIAS_GELU_BF16 = 1
ELIS_EPI_BIAS_RES_F32 = 2

KERNEL_CLASSES = ("seqmap", "embed_ln", "gemm_qkv", "attention", "gemm_o", "layernorm", "gemm_ffn1",
                  "gemm_ffn2", "pool_head", "select", "jobs")
K = {name: i for i, name in enumerate(KERNEL_CLASSES)}


class ElisLibraryMissing(RuntimeError):
    pass


class ElisError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        super().__init__(f"{where}: {elis_status_string(status)} ({status})")


class elis_config(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("d_ff", c_int32),
                ("vocab", c_int32), ("max_pos", c_int32), ("pooling", c_int32), ("head_hidden", c_int32),
                ("head_layers", c_int32), ("head_act", c_int32),
                ("ln_eps", c_float), ("out_scale", c_float), ("out_shift", c_float)]


class elis_layer_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("w_qkv", "w_o", "w_1", "w_2", "b_qkv", "b_o", "b_1", "b_2",
                                        "ln1_g", "ln1_b", "ln2_g", "ln2_b")]


class elis_weights(ctypes.Structure):
    _fields_ = [("cfg", elis_config), ("word", c_void_p), ("pos", c_void_p), ("type0", c_void_p),
                ("emb_ln_g", c_void_p), ("emb_ln_b", c_void_p), ("layers", POINTER(elis_layer_weights)),
                ("head_w1", c_void_p), ("head_b1", c_void_p), ("head_w2", c_void_p), ("head_b2", c_void_p),
                ("head_mid_w", POINTER(c_void_p)), ("head_mid_b", POINTER(c_void_p))]


class elis_job_table(ctypes.Structure):
    _fields_ = [("base", c_void_p), ("max_jobs", c_int32), ("max_pos", c_int32)]


# name -> (restype, argtypes); mirrors include/elis.h
SIGNATURES = {
    "elis_abi_version": (c_int32, []),
    "elis_status_string": (ctypes.c_char_p, [c_int]),
    "elis_predict_workspace_bytes": (c_size_t, [POINTER(elis_config), c_int32, c_int32, c_int32]),
    "elis_predict_remaining": (c_int, [POINTER(elis_weights), c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                       c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "elis_select_max_n": (c_int32, []),
    "elis_select_max_batch_cap": (c_int32, [c_int32]),
    "elis_select_workspace_bytes": (c_size_t, [c_int32]),
    "elis_isrtf_select": (c_int, [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p, c_void_p, c_size_t,
                                  c_void_p]),
    "elis_isrtf_select_noalloc": (c_int, [c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p, c_void_p]),
    "elis_read_status": (c_int, [c_void_p, c_void_p, POINTER(c_uint32)]),
    "elis_linear": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32, c_void_p,
                            c_void_p]),
    "elis_linear_plan": (c_int, [c_int32, c_int32, c_int32, c_int32, POINTER(c_int32)]),
    "elis_linear_with_plan": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32,
                                      POINTER(c_int32), c_void_p, c_void_p]),
    "elis_attention_workspace_bytes": (c_size_t, [c_int32, c_int32]),
    "elis_attention": (c_int, [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                               c_size_t, c_void_p]),
    "elis_layernorm": (c_int, [c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_float, c_void_p, c_void_p,
                               c_void_p]),
    "elis_pool_head_workspace_bytes": (c_size_t, [POINTER(elis_config), c_int32, c_int32]),
    "elis_pool_head": (c_int, [POINTER(elis_weights), c_void_p, c_void_p, c_int32, c_int32, c_int32, c_void_p,
                               c_void_p, c_size_t, c_void_p]),
    "elis_jobs_table_bytes": (c_size_t, [c_int32, c_int32]),
    "elis_jobs_init": (c_int, [POINTER(elis_job_table), c_void_p]),
    "elis_jobs_start": (c_int, [POINTER(elis_job_table), c_void_p, c_void_p, c_int32, c_void_p]),
    "elis_jobs_append": (c_int, [POINTER(elis_job_table), c_void_p, c_void_p, c_void_p, c_int32, c_int32,
                                 c_void_p]),
    "elis_jobs_pack": (c_int, [POINTER(elis_job_table), c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                               c_void_p]),
    "elis_jobs_store_pred": (c_int, [POINTER(elis_job_table), c_void_p, c_void_p, c_int32, c_void_p]),
    "elis_jobs_select_workspace_bytes": (c_size_t, [c_int32]),
    "elis_jobs_select": (c_int, [POINTER(elis_job_table), c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                                 c_void_p, c_size_t, c_void_p]),
    "elis_jobs_select_aged": (c_int, [POINTER(elis_job_table), c_void_p, c_void_p, c_float, c_int32, c_int32,
                                      c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "elis_timing_enable": (c_int, [c_uint32]),
    "elis_timing_stride": (c_int, [c_int32]),
    "elis_timing_reset": (c_int, []),
    "elis_timing_read": (c_int, [c_int32, POINTER(c_int32), POINTER(c_double)]),
}

_lib = None


def lib():
    """The loaded libelis.so (raises ElisLibraryMissing when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ElisLibraryMissing(f"{LIB_PATH} not found: build it with `python -m paper_2505_09142_amd.build`")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def elis_abi_version() -> int:
    return lib().elis_abi_version()


def elis_status_string(status: int) -> str:
    return lib().elis_status_string(status).decode()


def elis_predict_workspace_bytes(cfg: elis_config, total_tokens: int, n_seqs: int, max_seqlen: int) -> int:
    return lib().elis_predict_workspace_bytes(ctypes.byref(cfg), total_tokens, n_seqs, max_seqlen)


def elis_predict_remaining(w: elis_weights, token_ids: int, cu_seqlens: int, n_seqs: int, total_tokens: int,
                           max_seqlen: int, out_pred: int, out_hidden: int | None, workspace: int, ws_bytes: int,
                           stream: int | None) -> int:
    return lib().elis_predict_remaining(ctypes.byref(w) if w is not None else None, token_ids, cu_seqlens, n_seqs,
                                        total_tokens, max_seqlen, out_pred, out_hidden, workspace, ws_bytes, stream)


def elis_select_max_n() -> int:
    return lib().elis_select_max_n()


def elis_select_max_batch_cap(n: int) -> int:
    return lib().elis_select_max_batch_cap(n)


def elis_select_workspace_bytes(n: int) -> int:
    return lib().elis_select_workspace_bytes(n)


def elis_isrtf_select(pred: int, arrival_seq: int, n: int, batch_cap: int, out_idx: int, out_count: int,
                      workspace: int, ws_bytes: int, stream: int | None) -> int:
    return lib().elis_isrtf_select(pred, arrival_seq, n, batch_cap, out_idx, out_count, workspace, ws_bytes, stream)


ELIS_SELECT_NOALLOC_MAX_N = 1 << 18
ELIS_SELECT_NOALLOC_SCRATCH_BYTES = 3 << 20


def elis_isrtf_select_noalloc(pred: int, arrival_seq: int, n: int, batch_cap: int, out_idx: int, out_count: int,
                              stream: int | None) -> int:
    return lib().elis_isrtf_select_noalloc(pred, arrival_seq, n, batch_cap, out_idx, out_count, stream)


def elis_read_status(workspace: int, stream: int | None):
    """Returns (status, bits)."""
    bits = c_uint32(0)
    st = lib().elis_read_status(workspace, stream, ctypes.byref(bits))
    return st, bits.value


def elis_linear(x: int, w: int, bias: int, residual: int | None, m: int, n: int, k: int, epilogue: int, out: int,
                stream: int | None) -> int:
    return lib().elis_linear(x, w, bias, residual, m, n, k, epilogue, out, stream)


def elis_linear_with_plan(x: int, w: int, bias: int, residual: int | None, m: int, n: int, k: int, epilogue: int,
                          plan, out: int, stream: int | None) -> int:
    p = (c_int32 * 7)(*plan) if plan is not None else None
    return lib().elis_linear_with_plan(x, w, bias, residual, m, n, k, epilogue, p, out, stream)


def elis_linear_plan(m: int, n: int, k: int, epilogue: int):
    """Returns (status, (main_bm, main_bn, main_wgs, m1, rest_bm, rest_bn, rest_wgs))."""
    out = (c_int32 * 7)()
    st = lib().elis_linear_plan(m, n, k, epilogue, out)
    return st, tuple(out)


def elis_attention_workspace_bytes(n_seqs: int, total_tokens: int) -> int:
    return lib().elis_attention_workspace_bytes(n_seqs, total_tokens)


def elis_attention(qkv: int, cu_seqlens: int, n_seqs: int, total_tokens: int, max_seqlen: int, n_heads: int,
                   d_head: int, out: int, workspace: int, ws_bytes: int, stream: int | None) -> int:
    return lib().elis_attention(qkv, cu_seqlens, n_seqs, total_tokens, max_seqlen, n_heads, d_head, out, workspace,
                                ws_bytes, stream)


def elis_layernorm(x: int, g: int, b: int, rows: int, d: int, eps: float, out_f32: int | None,
                   out_bf16: int | None, stream: int | None) -> int:
    return lib().elis_layernorm(x, g, b, rows, d, eps, out_f32, out_bf16, stream)


def elis_pool_head_workspace_bytes(cfg: elis_config, n_seqs: int, max_seqlen: int) -> int:
    return lib().elis_pool_head_workspace_bytes(ctypes.byref(cfg), n_seqs, max_seqlen)


def elis_pool_head(w: elis_weights, hidden: int, cu_seqlens: int, n_seqs: int, total_tokens: int, max_seqlen: int,
                   out_pred: int, workspace: int, ws_bytes: int, stream: int | None) -> int:
    return lib().elis_pool_head(ctypes.byref(w) if w is not None else None, hidden, cu_seqlens, n_seqs,
                                total_tokens, max_seqlen, out_pred, workspace, ws_bytes, stream)


def _tab(t):
    return ctypes.byref(t) if t is not None else None


def elis_jobs_table_bytes(max_jobs: int, max_pos: int) -> int:
    return lib().elis_jobs_table_bytes(max_jobs, max_pos)


def elis_jobs_init(t: elis_job_table, stream: int | None) -> int:
    return lib().elis_jobs_init(_tab(t), stream)


def elis_jobs_start(t: elis_job_table, slots: int, arrival_seq: int, m: int, stream: int | None) -> int:
    return lib().elis_jobs_start(_tab(t), slots, arrival_seq, m, stream)


def elis_jobs_append(t: elis_job_table, slots: int, tok_offsets: int, tokens: int | None, m: int, total_new: int,
                     stream: int | None) -> int:
    return lib().elis_jobs_append(_tab(t), slots, tok_offsets, tokens, m, total_new, stream)


def elis_jobs_pack(t: elis_job_table, slots: int, n: int, total_tokens: int, max_seqlen: int, out_token_ids: int,
                   out_cu_seqlens: int, stream: int | None) -> int:
    return lib().elis_jobs_pack(_tab(t), slots, n, total_tokens, max_seqlen, out_token_ids, out_cu_seqlens, stream)


def elis_jobs_store_pred(t: elis_job_table, slots: int, pred: int, n: int, stream: int | None) -> int:
    return lib().elis_jobs_store_pred(_tab(t), slots, pred, n, stream)


def elis_jobs_select_workspace_bytes(a: int) -> int:
    return lib().elis_jobs_select_workspace_bytes(a)


def elis_jobs_select(t: elis_job_table, slots: int, a: int, batch_cap: int, out_slots: int | None, out_count: int,
                     workspace: int, ws_bytes: int, stream: int | None) -> int:
    return lib().elis_jobs_select(_tab(t), slots, a, batch_cap, out_slots, out_count, workspace, ws_bytes, stream)


def elis_jobs_select_aged(t: elis_job_table, slots: int, wait: int, aging: float, a: int, batch_cap: int,
                          out_slots: int | None, out_count: int, workspace: int, ws_bytes: int,
                          stream: int | None) -> int:
    return lib().elis_jobs_select_aged(_tab(t), slots, wait, aging, a, batch_cap, out_slots, out_count, workspace,
                                       ws_bytes, stream)


def elis_timing_enable(class_mask: int) -> int:
    return lib().elis_timing_enable(class_mask)


def elis_timing_stride(every: int) -> int:
    return lib().elis_timing_stride(every)


def elis_timing_reset() -> int:
    return lib().elis_timing_reset()


def elis_timing_read(kernel_class: int):
    """Returns (status, launches, total_ms)."""
    n = c_int32(0)
    ms = c_double(0.0)
    st = lib().elis_timing_read(kernel_class, ctypes.byref(n), ctypes.byref(ms))
    return st, n.value, ms.value


def check(status: int, where: str = "") -> None:
    if status != ELIS_OK:
        raise ElisError(status, where)
