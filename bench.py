#!/usr/bin/env python3
"""Throughput of the ELIS hot path on one MI355X.

One step = one scheduling round over a resident batch: elis_predict_remaining
(BERT-base-shaped encoder + CLS pooling + 768->256->1 head over 64 packed
in-flight sequences) followed by elis_isrtf_select (batch_cap 32). Inputs and
weights are in HBM before the timed region starts.

Prints ONE JSON line. `value` is predicted sequences per second; tokens/s and
the p50/p99 predict+select latency per round ride along. `roofline` is for the
kernel class with the largest share of GPU time, timed live over the timed
region with HIP events on the launch stream (the library's opt-in timing);
`cpu_baseline` is the fp64 oracle on a bounded sample of the same batch.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def _algorithmic(w, b):
    """Per-launch algorithmic FLOPs (contractions) or bytes (row kernels) by kernel class."""
    s = w.shape
    T, n, d, F, L = b.total, b.n, s.d_model, s.d_ff, s.n_layers
    sumsq = float((b.lengths.astype(float) ** 2).sum())
    return {
        "gemm_qkv": ("flop", 2.0 * T * d * 3 * d, L),
        "attention": ("flop", 4.0 * sumsq * d, L),
        "gemm_o": ("flop", 2.0 * T * d * d, L),
        "gemm_ffn1": ("flop", 2.0 * T * d * F, L),
        "gemm_ffn2": ("flop", 2.0 * T * F * d, L),
        # fp32 row in; fp32 + bf16 rows out (the last LayerNorm writes fp32 only: counted as the common case)
        "layernorm": ("byte", T * d * (4.0 + 4.0 + 2.0), 2 * L),
        # ids + gathered bf16 word and position rows in; fp32 + bf16 rows out
        "embed_ln": ("byte", T * (4.0 + d * (2.0 + 2.0 + 4.0 + 2.0)), 1),
        "pool_head": ("byte", n * d * 4.0 + (s.head_hidden or 1) * d * 4.0, 1),
        "seqmap": ("byte", (n + 1) * 4.0 * 4, 1),
        "select": ("byte", n * 12.0 + w.batch_cap * 4.0, 1),
    }


def _source_sha(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _traffic(kernel_class: str):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, if the kernel source is unchanged."""
    path = os.path.join(ROOT, "profiles", f"{kernel_class}_bert_base_b64_traffic.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"^traffic:\s*(\{.*\})\s*$", open(path).read(), re.M)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != _source_sha(rec.get("sources", [])):
        return None
    return rec.get("per_launch_bytes")


def cpu_baseline(w, W, b, seconds: float):
    import numpy as np
    import threadpoolctl

    import oracle
    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()), default=1)
    t0 = time.perf_counter()
    done, toks = 0, 0
    while done < b.n and (time.perf_counter() - t0) < seconds:
        s = done
        oracle.oracle_forward(b.token_ids, b.cu_seqlens, W.master, w.shape, want_hidden=False, seqs=[s])
        done += 1
        toks += int(b.lengths[s])
    oracle.oracle_select(np.zeros(b.n, np.float32), b.arrival_seq, w.batch_cap)
    el = time.perf_counter() - t0
    return {"value": done / el, "unit": "seqs/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {done} of {b.n} sequences ({toks} tokens) of the same batch, fp64 numpy encoder "
                      f"+ sort-based select, {el:.1f} s",
            "tokens_per_s": toks / el, "host_cpus": len(os.sched_getaffinity(0))}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="bert_base_b64")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the hot path is single-GPU by design); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2505_09142_amd import _elis as E
    from paper_2505_09142_amd.device import DeviceWeights, Predictor, upload_batch
    from workloads import WORKLOADS, make_batch, make_weights

    w = WORKLOADS[args.workload]
    W = make_weights(w.shape, w.weight_seed)
    b = make_batch(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    pr = Predictor(DeviceWeights(w.shape, W.device, dev), dev)
    ids, cu, arr = upload_batch(b, dev)
    pred = torch.empty(b.n, dtype=torch.float32, device=dev)
    out_idx = torch.empty(max(1, w.batch_cap), dtype=torch.int32, device=dev)
    out_cnt = torch.empty(1, dtype=torch.int32, device=dev)
    T, n, msl = b.total, b.n, b.max_seqlen

    def step():
        pr.predict(ids, cu, msl, out_pred=pred)
        pr.select(pred, arr, w.batch_cap, out_idx, out_cnt)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    st, bits = pr.status()
    if st != E.ELIS_OK:
        raise SystemExit(f"device status {st} bits {bits}")

    # Per-class breakdown (events around every launch), to find the dominant kernel.
    alg = _algorithmic(w, b)
    E.elis_timing_reset()
    E.elis_timing_enable((1 << len(E.KERNEL_CLASSES)) - 1)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    E.elis_timing_enable(0)
    kernels = {}
    for name in E.KERNEL_CLASSES:
        s_, nl, ms = E.elis_timing_read(E.K[name])
        if nl == 0:
            continue
        kind, per_launch, _ = alg[name]
        avg_s = ms / nl * 1e-3
        rate = per_launch / avg_s / (1e12 if kind == "flop" else 1e9)
        kernels[name] = {"launches_per_step": nl / args.steps, "avg_us": avg_s * 1e6, "ms_per_step": ms / args.steps,
                         ("tflops" if kind == "flop" else "gbs"): rate}
    dominant = max(kernels, key=lambda k: kernels[k]["ms_per_step"])

    # Timed region: events around the dominant class only, plus per-step events.
    E.elis_timing_reset()
    E.elis_timing_enable(1 << E.K[dominant])
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        evs[i][0].record()
        step()
        evs[i][1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    E.elis_timing_enable(0)
    _, dl, dms = E.elis_timing_read(E.K[dominant])
    elapsed = t1 - t0
    lat = np.array([a.elapsed_time(c) for a, c in evs])
    st, bits = pr.status()
    if st != E.ELIS_OK:
        raise SystemExit(f"device status {st} bits {bits}")

    kind, per_launch, _ = alg[dominant]
    avg_s = dms / dl * 1e-3
    if kind == "flop":
        achieved, peak, unit, bound = per_launch / avg_s / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s", "mfma"
    else:
        achieved, peak, unit, bound = per_launch / avg_s / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
    gemm_flop = sum(alg[k][1] * alg[k][2] for k in ("gemm_qkv", "gemm_o", "gemm_ffn1", "gemm_ffn2"))
    gemm_s = sum(kernels[k]["ms_per_step"] for k in ("gemm_qkv", "gemm_o", "gemm_ffn1", "gemm_ffn2")) * 1e-3
    att_s = kernels["attention"]["ms_per_step"] * 1e-3
    att_flop = alg["attention"][1] * alg["attention"][2]

    out = {
        "metric": "predicted seqs/sec + tokens/sec per round; MFMA util; p50 predict+select latency",
        "value": n * args.steps / elapsed,
        "unit": "seqs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: BERT-base-shaped predictor (12 layers, d_model 768, 12 heads, FFN 3072, "
                               f"CLS pooling, 768->256->1 head), {n} packed in-flight sequences, ISRTF select "
                               f"{w.batch_cap} of {n}",
                   "n_seqs": n, "total_tokens": T, "max_seqlen": msl, "batch_cap": w.batch_cap,
                   "global_batch": n, "seq_len": msl, "parallelism": "none (1 GPU)"},
        "tokens_per_s": T * args.steps / elapsed,
        "p50_ms": float(np.percentile(lat, 50)),
        "p99_ms": float(np.percentile(lat, 99)),
        "mfma_util_gemm": gemm_flop / gemm_s / 1e12 / PEAK_BF16_TFLOPS,
        "mfma_util_attention": att_flop / att_s / 1e12 / PEAK_BF16_TFLOPS,
        "roofline": {"bound": bound, "kernel": dominant, "achieved": achieved, "peak": peak, "unit": unit,
                     "frac": achieved / peak, "traffic": _traffic(dominant),
                     "per_launch_" + ("flop" if kind == "flop" else "bytes"): per_launch,
                     "avg_launch_us": avg_s * 1e6, "launches": dl},
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, W, b, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
