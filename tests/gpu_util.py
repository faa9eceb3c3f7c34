"""Helpers shared by the GPU tests (device plumbing only; no oracle arithmetic)."""
import sys

import numpy as np
import torch

from paper_2505_09142_amd import _elis as E


def note(msg: str) -> None:
    """Print and flush a line naming the case about to run on the GPU."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


def host_u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def workspace(nbytes: int):
    buf = torch.empty(max(256, nbytes) + 256, dtype=torch.uint8, device="cuda")
    base = buf.data_ptr()
    al = (base + 255) // 256 * 256
    return buf, al, buf.numel() - (al - base)


def ok(status: int, what: str = "") -> None:
    assert status == E.ELIS_OK, f"{what}: {E.elis_status_string(status)}"
