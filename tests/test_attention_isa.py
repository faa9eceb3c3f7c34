"""The d_head-64 attention kernel's tile pipeline, checked in the compiled code (CPU only).

Each key tile's K and V go from global memory straight into LDS, the next tile's loads are
issued into the other buffer right after the tile's barrier, and they are waited for (one
explicit vmcnt wait) only before the next barrier. The compiler tracks such direct-to-LDS
loads by LDS variable: when both buffers were one array it could not tell the buffer being
loaded from the one being read, and put a vmcnt(0) wait before the first LDS read of every
tile, so each tile waited out the next one's loads. This test compiles attention.hip for gfx950
with the library's flags and checks, in the all-queries kernel and the CLS-only one, that between
a direct-to-LDS load and the next barrier no LDS read is preceded by a vmcnt wait.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2505_09142_amd import build as B

KERNELS = {  # all queries; the CLS-only tail of the last layer
    "all": "_ZN4elis12_GLOBAL__N_116attention_kernelILi64ELb0EEEvPKtPKiS5_S5_iPtfi",
    "cls": "_ZN4elis12_GLOBAL__N_116attention_kernelILi64ELb1EEEvPKtPKiS5_S5_iPtfi",
}
DMA = re.compile(r"^\s*(buffer_load_dword\S*\s.*\blds\b|global_load_lds_dword\S*)")
WAIT = re.compile(r"^\s*s_waitcnt\s.*vmcnt\(")
READ = re.compile(r"^\s*ds_read")
BARRIER = re.compile(r"^\s*s_barrier\b")


def kernel_asm(tmp_path, kernel):
    if not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    src = os.path.join(B.CSRC, "attention.hip")
    out = tmp_path / "attention.s"
    cmd = [B.HIPCC, *B.CFLAGS, *B.EXTRA["attention.hip"], "--cuda-device-only", "-S", src, "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = out.read_text().split("\n")
    start = next(i for i, l in enumerate(lines) if l.startswith(kernel + ":"))
    end = next(i for i in range(start, len(lines)) if lines[i].strip().startswith("s_endpgm"))
    return lines[start:end]


LABEL = re.compile(r"^(\.LBB\w+):")
BRANCH = re.compile(r"^\s*(s_branch|s_cbranch_\w+)\s+(\.LBB\w+)")


def blocks(body):
    """Basic blocks of the function: (instructions, successor labels, falls through)."""
    out, cur, name = {}, [], "entry"
    order = []
    def close(nxt_fall):
        order.append(name)
        out[name] = (cur, succ, nxt_fall)
    succ = []
    for line in body[1:]:
        m = LABEL.match(line)
        if m:
            close(True)
            name, cur, succ = m.group(1), [], []
            continue
        ins = line.split(";")[0].strip()
        if not ins or ins.startswith("."):
            continue
        cur.append(ins)
        b = BRANCH.match(ins)
        if b:
            succ.append(b.group(2))
            uncond = b.group(1) == "s_branch"
            close(not uncond)
            name, cur, succ = f"{name}+", [], []
    close(False)
    # successor lists with fall-through to the next block in layout order
    cfg = {}
    for i, n in enumerate(order):
        ins, sc, fall = out[n]
        nxt = list(sc)
        if fall and i + 1 < len(order):
            nxt.append(order[i + 1])
        cfg[n] = (ins, nxt)
    return order, cfg


@pytest.mark.parametrize("which", sorted(KERNELS))
def test_no_wait_on_tile_loads_before_lds_reads(tmp_path, which):
    body = kernel_asm(tmp_path, KERNELS[which])
    assert any(DMA.match(l) for l in body), "no direct-to-LDS loads found"
    order, cfg = blocks(body)
    # Forward dataflow over the control-flow graph. State bits: A = a direct-to-LDS load was
    # issued since the last barrier; W = a vmcnt wait followed it. An LDS read under W is a wait
    # on in-flight tile loads before the tile's own reads.
    state_in = {n: 0 for n in order}
    work = list(order)
    bad = set()
    while work:
        n = work.pop(0)
        st = state_in[n]
        ins, nxt = cfg[n]
        for x in ins:
            if BARRIER.match(x):
                st = 0
            elif DMA.match(x):
                st |= 1
            elif WAIT.match(x) and st & 1:
                st |= 2
            elif READ.match(x) and st & 2:
                bad.add((n, x))
        for m in nxt:
            if m in state_in and (state_in[m] | st) != state_in[m]:
                state_in[m] |= st
                work.append(m)
    assert not bad, f"LDS reads behind a vmcnt wait on in-flight tile loads: {sorted(bad)[:3]}"
