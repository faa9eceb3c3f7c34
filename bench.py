#!/usr/bin/env python3
"""Throughput of the ELIS hot path on one MI355X.

One step = one scheduling round over a resident batch: elis_predict_remaining
(BERT-base-shaped encoder + CLS pooling + 768->256->1 head over 64 packed
in-flight sequences) followed by elis_isrtf_select (batch_cap 32). Inputs and
weights are in HBM before the timed region starts.

Prints ONE JSON line. `value` is predicted sequences per second; tokens/s and
the p50/p99 predict+select latency per round ride along. `roofline` is for the
kernel class with the largest share of GPU time, timed live over the timed
region with HIP events attached to its dispatches on the launch stream (the
library's opt-in timing, on every 13th launch of the class);
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


def _head_params(s):
    nl, hh, d = s.n_head_layers, s.head_hidden, s.d_model
    if nl == 1:
        return d + 1
    return hh * d + hh + (nl - 2) * (hh * hh + hh) + hh + 1


def _describe(w):
    s = w.shape
    pool = "CLS" if s.pooling == 0 else "mean"
    if s.n_head_layers == 1:
        head = f"{s.d_model}->1"
    elif s.n_head_layers == 2:
        head = f"{s.d_model}->{s.head_hidden}->{'ReLU' if s.head_act == 0 else 'linear'}->1"
    else:
        head = (f"{s.n_head_layers} FC layers, width {s.head_hidden}, "
                f"{'ReLU' if s.head_act == 0 else 'no activation'}")
    return (f"{w.name}: {s.name}-shaped predictor ({s.n_layers} layers, d_model {s.d_model}, {s.n_heads} heads, "
            f"FFN {s.d_ff}, {pool} pooling, head {head}), {w.n_seqs} packed in-flight sequences, ISRTF select "
            f"{w.batch_cap} of {w.n_seqs}")


def _algorithmic(w, b):
    """Algorithmic FLOPs (contractions) or bytes (row kernels) by kernel class: (kind, the work of
    each launch of one step in launch order, launches per step). With CLS pooling the last layer
    needs, after its QKV product, only the CLS rows (one attention query and one row of every later
    product per sequence); that is all the library computes there, and all that is counted."""
    s = w.shape
    T, n, d, F, L = b.total, b.n, s.d_model, s.d_ff, s.n_layers
    lens = b.lengths.astype(float)
    sumsq = float((lens ** 2).sum())
    cls_tail = s.pooling == 0 and L > 0
    rows = [T] * L
    att = [4.0 * d * sumsq] * L
    if cls_tail:
        rows[-1] = n
        att[-1] = 4.0 * d * float(lens.sum())
    # fp32 row in; bf16 row + (mean, rstd) out (the last LayerNorm writes an fp32 row instead:
    # counted as the common case)
    ln_row = d * (4.0 + 2.0) + 8.0
    ln = [r * ln_row for r in rows for _ in (0, 1)]  # after the out-projection and after FFN2
    alg = {
        "gemm_qkv": ("flop", [2.0 * T * d * 3 * d] * L),
        "attention": ("flop", att),
        "gemm_o": ("flop", [2.0 * r * d * d for r in rows]),
        "gemm_ffn1": ("flop", [2.0 * r * d * F for r in rows]),
        "gemm_ffn2": ("flop", [2.0 * r * F * d for r in rows]),
        "layernorm": ("byte", ln),
        # ids + gathered bf16 word and position rows in; fp32 pre-norm + bf16 rows + stats out
        "embed_ln": ("byte", [T * (4.0 + d * (2.0 + 2.0 + 4.0 + 2.0) + 8.0)]),
        # the hidden rows pooling reads (CLS: one per sequence; mean: every token) + every head weight once
        "pool_head": ("byte", [(n if s.pooling == 0 else T) * d * 4.0 + 4.0 * _head_params(s)]),
        "seqmap": ("byte", [(n + 1) * 4.0 * 4]),
        "select": ("byte", [n * 12.0 + w.batch_cap * 4.0]),
    }
    return {k: (kind, per, len(per)) for k, (kind, per) in alg.items() if per}


def sampled_work(per_launch, stride, launches):
    """Average work of the launches a stride-`stride` sample timed: launch j = stride * i of the
    class since the reset, i < launches, is launch j mod (launches per step) of its step."""
    m = len(per_launch)
    return sum(per_launch[(stride * i) % m] for i in range(launches)) / launches


def _source_sha(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "bert_base_b64_hbm_traffic.md")

# Kernels behind each class at a workload, and the sources whose text fixes them: a PMC figure
# is reported only while those sources are unchanged. A GEMM class is one launch or two (the
# library's launch plan may split the rows between a large-tile and a small-tile launch); the
# plan comes from elis_linear_plan at the workload's token count.
_GEMM_SRC = ["paper_2505_09142_amd/csrc/gemm.hip", "paper_2505_09142_amd/csrc/gemm_common.h",
             "paper_2505_09142_amd/csrc/common.h", "paper_2505_09142_amd/csrc/kernels.h"]
_GEMM_EPI = {"gemm_qkv": (0, 0), "gemm_o": (2, 4), "gemm_ffn1": (1, 1), "gemm_ffn2": (2, 5)}  # public, internal


def _gemm_kernel(bm, bn, wgs, epi, n, f32):
    if (bm, bn) == (256, 256):
        return f"gemm_sched_kernel<256, 256, 2, 4, 32, {epi}, 1, 2>"
    if (bm, bn) == (128, 128):
        return f"gemm_sched_kernel<128, 128, 2, 2, 32, {epi}, 2, 2>"
    if (bm, bn) == (64, 128):
        return f"gemm_sched_kernel<64, 128, 2, 2, 32, {epi}, {wgs}, {2 if wgs == 2 else 4}>"
    if (bm, bn) == (64, 64):
        return f"gemm_sched_kernel<64, 64, 2, 2, 32, {epi}, {wgs}, {2 if wgs == 4 else 4}>"
    return f"gemm_kernel<128, 64, 2, 2, 16, {epi}>"


def class_kernels(workload: str) -> dict:
    """class -> (kernel names any launch of the class dispatches, sources, launches per pass).
    A GEMM class uses the plan at T rows (one or two kernels) and, with CLS pooling, the plan at
    n rows in the last layer; the out-projection of that layer also gathers its residual rows."""
    from paper_2505_09142_amd import _elis as E
    from workloads import WORKLOADS, make_batch
    w = WORKLOADS[workload]
    s = w.shape
    b = make_batch(w)
    T, n, d, F, L = b.total, b.n, s.d_model, s.d_ff, s.n_layers
    cls_tail = s.pooling == 0 and L > 0
    dims = {"gemm_qkv": (3 * d, d), "gemm_o": (d, d), "gemm_ffn1": (F, d), "gemm_ffn2": (d, F)}
    out = {}
    for cls, (nn, k) in dims.items():
        pub, internal = _GEMM_EPI[cls]
        names = []
        for m in ([T, n] if cls_tail and cls != "gemm_qkv" else [T]):
            st, (bm, bn, wg, m1, rbm, rbn, rwg) = E.elis_linear_plan(m, nn, k, pub)
            if st != 0:
                raise SystemExit(f"elis_linear_plan failed for {cls}: {st}")
            for kname in [_gemm_kernel(bm, bn, wg, internal, nn, pub == 2)] + (
                    [_gemm_kernel(rbm, rbn, rwg, internal, nn, pub == 2)] if m1 < m else []):
                if kname not in names:
                    names.append(kname)
        if cls == "gemm_o" and cls_tail:
            names.append("gather_rows_kernel")
        out[cls] = (names, _GEMM_SRC, L)
    vpl = (d + 255) // 256
    att = [f"attention_kernel<{d // s.n_heads}, false>"] + ([f"attention_kernel<{d // s.n_heads}, true>"] if cls_tail
                                                             else [])
    out["attention"] = (att, ["paper_2505_09142_amd/csrc/attention.hip", "paper_2505_09142_amd/csrc/common.h"], L)
    out["layernorm"] = ([f"layernorm_kernel<{vpl}>"], ["paper_2505_09142_amd/csrc/norm.hip",
                                                        "paper_2505_09142_amd/csrc/common.h"], 2 * L)
    return out


COPY_KERNEL = "__amd_rocclr_copyBuffer"


def _traffic(kernel_class: str):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, if the kernel source is unchanged."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    m = re.search(r"^traffic\[" + re.escape(kernel_class) + r"\]:\s*(\{.*\})\s*$", open(TRAFFIC_PROFILE).read(), re.M)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != _source_sha(rec.get("sources", [])):
        return None
    return rec.get("per_launch_bytes")


def _pmc_per_kernel(csv_path, counter):
    """Counter values (KiB) per dispatch, grouped by demangled kernel name."""
    import csv
    import collections
    out = collections.defaultdict(list)
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"].replace("elis::(anonymous namespace)::", "").replace("void ", "")
            out[re.sub(r"\(.*", "", name).strip()].append(float(r["Counter_Value"]))
    return out


def summarize_pmc(fetch_csv, write_csv, copy_mib, workload, commands):
    """Write the HBM-traffic summary from one FETCH_SIZE and one WRITE_SIZE rocprofv3 pass.

    Each counter is scaled by bytes/KiB-reading of the plain device copy of copy_mib MiB
    that both passes ran first (the largest copy dispatches of each pass)."""
    from workloads import WORKLOADS, make_batch
    w = WORKLOADS[workload]
    b = make_batch(w)
    fetch = _pmc_per_kernel(fetch_csv, "FETCH_SIZE")
    write = _pmc_per_kernel(write_csv, "WRITE_SIZE")
    nbytes = copy_mib * 2 ** 20
    cf = sorted(fetch[COPY_KERNEL])[-3:]
    cw = sorted(write[COPY_KERNEL])[-3:]
    f_scale = nbytes / (sum(cf) / len(cf) * 1024)
    w_scale = nbytes / (sum(cw) / len(cw) * 1024)
    T, n, d, F, L = b.total, b.n, w.shape.d_model, w.shape.d_ff, w.shape.n_layers
    cls_tail = w.shape.pooling == 0 and L > 0

    def mand(r):  # bytes a launch over r rows must move at least once: operands in, results out
        return {
            "gemm_o": r * d * 2 + d * d * 2 + d * 4 * 3 + r * 8 + r * d * 4 * 2,
            "layernorm": r * (d * (4 + 2) + 8),
            "gemm_ffn1": r * d * 2 + F * d * 2 + F * 4 + r * F * 2,
            "gemm_ffn2": r * F * 2 + F * d * 2 + d * 4 * 3 + r * 8 + r * d * 4 * 2,
        }
    full, tail = mand(T), mand(n if cls_tail else T)
    qkv_b = T * 3 * d * 2
    mandatory = {c: ((L - 1) * full[c] + tail[c]) / L for c in full}  # average over the layers
    mandatory["gemm_qkv"] = T * d * 2 + 3 * d * d * 2 + 3 * d * 4 + qkv_b
    att_tail = (qkv_b * 2 // 3 + n * d * 2 * 2) if cls_tail else qkv_b + T * d * 2
    mandatory["attention"] = ((L - 1) * (qkv_b + T * d * 2) + att_tail) / L
    passes = len(fetch.get("seqmap_kernel", []))
    lines = [f"# HBM traffic per launch: {workload} (T = {T:,}), rocprofv3 PMC byte counters", "",
             "Two passes over the same bench command, one counter each (MI355X, repo root as working tree):", ""]
    lines += [f"    {c}" for c in commands]
    lines += ["", f"Scale: before its steps each pass runs a plain device-to-device copy of {copy_mib} MiB "
              f"three times (`{COPY_KERNEL}`). Counter readings of those copies: FETCH_SIZE "
              f"{', '.join(f'{v:.0f}' for v in cf)} KiB, WRITE_SIZE {', '.join(f'{v:.0f}' for v in cw)} KiB, "
              f"for {nbytes / 1024:.0f} KiB moved each way, so bytes = FETCH_SIZE x 1024 x {f_scale:.4f} "
              f"and WRITE_SIZE x 1024 x {w_scale:.4f}.", "",
              "| class | kernels | launches | FETCH_SIZE KiB / launch | WRITE_SIZE KiB / launch | scaled MB / launch | mandatory MB / launch | ratio |",
              "|---|---|---:|---:|---:|---:|---:|---:|"]
    recs = {}
    for cls, (knames, srcs, lpp) in class_kernels(workload).items():
        label = " + ".join(f"`{k}`" for k in knames)
        fvs, wvs = [fetch.get(k, []) for k in knames], [write.get(k, []) for k in knames]
        if not passes or not all(fvs) or not all(wvs):
            lines.append(f"| {cls} | {label} | 0 | - | - | - | - | - |")
            continue
        # per class launch: every dispatch of the class's kernels over the passes, / launches
        launches = passes * lpp
        fk = sum(sum(v) for v in fvs) / launches
        wk = sum(sum(v) for v in wvs) / launches
        tb = fk * 1024 * f_scale + wk * 1024 * w_scale
        lines.append(f"| {cls} | {label} | {launches} | {fk:,.0f} | {wk:,.0f} | {tb / 1e6:,.1f} | "
                     f"{mandatory[cls] / 1e6:,.1f} | {tb / mandatory[cls]:.2f} |")
        recs[cls] = {"per_launch_bytes": tb, "fetch_kib": fk, "write_kib": wk, "fetch_scale": f_scale,
                     "write_scale": w_scale, "mandatory_bytes": mandatory[cls], "kernels": knames,
                     "sources": srcs, "source_sha256": _source_sha(srcs)}
    lines += ["", "`ratio` = scaled traffic / mandatory bytes; above 1 means operands were fetched from "
              "memory more than once (tiles re-read after leaving L2).", "",
              "Machine-readable records (bench.py reads these; a record whose sources have changed since is ignored):", ""]
    lines += [f"traffic[{c}]: {json.dumps(r)}" for c, r in recs.items()]
    with open(TRAFFIC_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {TRAFFIC_PROFILE}")


MFMA_PROFILE = os.path.join(ROOT, "profiles", "bert_base_b64_mfma_busy.md")


def summarize_mfma(csv_path, bench_json, command):
    """MFMA busy fraction per kernel from one rocprofv3 --pmc pass with SQ_VALU_MFMA_BUSY_CYCLES and
    SQ_BUSY_CYCLES, next to bench.py's algorithmic utilisation from the same run."""
    import collections
    import csv
    rec = json.loads([x for x in open(bench_json) if x.startswith("{")][-1])
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    durations = collections.defaultdict(dict)  # kernel -> dispatch id -> ns (profiler timestamps)
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            n = re.sub(r"\(.*", "", r["Kernel_Name"].replace("elis::(anonymous namespace)::", "").replace("void ", "")).strip()
            vals[n][r["Counter_Name"]].append(float(r["Counter_Value"]))
            durations[n][r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    passes = len(durations.get("seqmap_kernel", {}))
    simds, ses = 1024, 32  # MI355X: 256 CUs x 4 SIMDs; 8 XCDs x 4 shader engines
    lines = ["# MFMA busy per kernel: bert_base_b64, rocprofv3 PMC counters", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             "busy = SQ_VALU_MFMA_BUSY_CYCLES / 1024 SIMDs ÷ (SQ_BUSY_CYCLES / 32 shader engines): the fraction of "
             "the kernel's busy cycles in which an average SIMD's matrix core was working. `algorithmic` = "
             "bench.py's FLOPs per launch ÷ the class's kernel time per launch ÷ 2.5 PFLOP/s, the time taken "
             f"from the dispatch timestamps of the same run ({passes} forward passes; bench.py's own HIP events "
             "also time the profiler's per-dispatch counter work under --pmc); the ratio algorithmic / busy is "
             "(clock under load) ÷ 2.4 GHz when the matrix cores run at their full rate while busy.", "",
             "| class | kernels | dispatches | MFMA busy | algorithmic | algorithmic / busy |",
             "|---|---|---:|---:|---:|---:|"]
    for cls, (knames, _, per_pass) in class_kernels(rec["config"]["workload"].split(":")[0]).items():
        vs = [vals.get(k) for k in knames]
        if not all(v and v.get("SQ_VALU_MFMA_BUSY_CYCLES") for v in vs):
            continue
        # cycles summed over every dispatch of the class's kernels
        mb = sum(sum(v["SQ_VALU_MFMA_BUSY_CYCLES"]) for v in vs)
        bc = sum(sum(v["SQ_BUSY_CYCLES"]) for v in vs)
        busy = mb / simds / (bc / ses)
        k = rec["kernels"].get(cls, {})
        alg = None
        if "tflops" in k and passes:
            flop = k["tflops"] * 1e12 * k["avg_us"] * 1e-6  # per launch, independent of its timing
            ns = sum(sum(durations[x].values()) for x in knames) / (passes * per_pass)
            alg = flop / (ns * 1e-9) / 1e12 / PEAK_BF16_TFLOPS
        label = " + ".join(f"`{x}`" for x in knames)
        lines.append(f"| {cls} | {label} | {sum(len(v['SQ_BUSY_CYCLES']) for v in vs)} | {busy:.3f} | "
                     + (f"{alg:.3f} | {alg / busy:.2f} |" if alg is not None and busy > 0 else "- | - |"))
    with open(MFMA_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {MFMA_PROFILE}")


ISSUE_PROFILE = os.path.join(ROOT, "profiles", "bert_base_b64_issue_counters.md")
ISSUE_COUNTERS = ("SQ_BUSY_CYCLES", "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_VALU_TRANS_F32",
                  "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", "SQ_ACTIVE_INST_VALU")


def summarize_issue(csv_path, command):
    """Instruction mix and LDS bank conflicts per kernel class from one rocprofv3 --pmc pass
    with ISSUE_COUNTERS (summed over every dispatch of the class's kernels)."""
    import collections
    import csv
    vals = collections.defaultdict(lambda: collections.defaultdict(float))
    disp = collections.defaultdict(set)
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            n = re.sub(r"\(.*", "", r["Kernel_Name"].replace("elis::(anonymous namespace)::", "").replace("void ", "")).strip()
            vals[n][r["Counter_Name"]] += float(r["Counter_Value"])
            disp[n].add(r["Dispatch_Id"])
    simds, ses = 1024, 32  # MI355X: 256 CUs x 4 SIMDs; 8 XCDs x 4 shader engines
    lines = ["# Instruction mix and LDS bank conflicts per kernel class: bert_base_b64, rocprofv3 PMC counters", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             "Counters summed over every dispatch of a class's kernels. `VALU / MFMA` = (SQ_INSTS_VALU − "
             "SQ_INSTS_MFMA) / SQ_INSTS_MFMA (SQ_INSTS_VALU counts the matrix instructions too); `trans / MFMA` "
             "= SQ_INSTS_VALU_TRANS_F32 / SQ_INSTS_MFMA. `VALU issue` = 4 cycles per non-matrix VALU "
             "instruction (a wave64 instruction on a 16-lane SIMD) ÷ 1024 SIMDs ÷ (SQ_BUSY_CYCLES / 32 shader "
             "engines): the fraction of the kernel's cycles an average SIMD's vector ALU spent issuing, "
             "transcendentals counted at one pass. `LDS conflicts` = SQ_LDS_BANK_CONFLICT / (SQ_LDS_IDX_ACTIVE − "
             "SQ_LDS_BANK_CONFLICT): bank-conflict stall cycles per active LDS cycle.", "",
             "| class | dispatches | VALU / MFMA | trans / MFMA | VALU issue | LDS conflicts |",
             "|---|---:|---:|---:|---:|---:|"]
    rec_cls = class_kernels("bert_base_b64")
    for cls, (knames, _, _) in rec_cls.items():
        vs = [vals.get(k) for k in knames]
        if not all(vs):
            continue
        tot = collections.defaultdict(float)
        for v in vs:
            for c, x in v.items():
                tot[c] += x
        mf = tot["SQ_INSTS_MFMA"]
        valu = tot["SQ_INSTS_VALU"] - mf
        cyc = tot["SQ_BUSY_CYCLES"] / ses
        issue = 4.0 * valu / simds / cyc if cyc else 0.0
        lds = tot["SQ_LDS_IDX_ACTIVE"] - tot["SQ_LDS_BANK_CONFLICT"]
        conf = tot["SQ_LDS_BANK_CONFLICT"] / lds if lds > 0 else 0.0
        lines.append(f"| {cls} | {sum(len(disp[k]) for k in knames)} | "
                     + (f"{valu / mf:.2f} | {tot['SQ_INSTS_VALU_TRANS_F32'] / mf:.2f}" if mf else "- | -")
                     + f" | {issue:.2f} | {conf:.3f} |")
    with open(ISSUE_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {ISSUE_PROFILE}")


TRACE_PROFILE = os.path.join(ROOT, "profiles", "bert_base_b64_kernel_trace.md")
_ROLES = {"seqmap_kernel": "sequence table", "embed_ln_kernel<3>": "embedding + LN",
          "select_rank_kernel": "ISRTF select", "head_tile_kernel<0, true, 8>": "head 768->256 + ReLU (CLS rows)",
          "head_out_kernel": "head 256->1, affine", COPY_KERNEL: "(torch copies)"}


def summarize_trace(stats_csv, command, bench_json, plain_json=None):
    """Write the kernel-trace summary from a rocprofv3 --stats kernel_stats.csv and the
    JSON line bench.py printed in the same run (plain_json: a line from a run without the
    profiler on the same box, whose HIP events carry no tracing work)."""
    import csv
    rec = json.loads(open(bench_json).read().strip().splitlines()[-1])
    roles = dict(_ROLES)
    ck = class_kernels(rec["config"]["workload"].split(":")[0])
    roles.update({k: c for c, (ks, _, _) in ck.items() for k in ks})
    rows, tot, calls = [], {}, {}
    with open(stats_csv) as f:
        for r in csv.DictReader(f):
            n = re.sub(r"\(.*", "", r["Name"].replace("elis::(anonymous namespace)::", "").replace("void ", "")).strip()
            tot[n] = float(r["TotalDurationNs"]) / 1e3
            calls[n] = int(r["Calls"])
            rows.append(f"| `{n}` | {roles.get(n, '')} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e3:.1f} | "
                        f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    rl = rec["roofline"]
    dom = rl["kernel"]
    passes = calls.get("seqmap_kernel", 0)
    prof_us = (sum(tot.get(k, 0.0) for k in ck[dom][0]) / (passes * ck[dom][2])
               if dom in ck and passes and all(k in tot for k in ck[dom][0]) else None)
    cfg = rec["config"]
    steps, warm = rec["steps"], rec["warmup"]
    lines = [f"# Kernel trace: {cfg['workload'].split(':')[0]} (T = {cfg['total_tokens']:,}), predict + select", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             f"{warm + 2 * steps} forward passes were traced ({warm} warm-up + {steps} per-class-timed + {steps} "
             "timed steps). Table from the `kernel_stats.csv` of that run.", "",
             "| kernel | class | calls | total µs | avg µs | % of GPU time |", "|---|---|---:|---:|---:|---:|"]
    lines += rows
    lines += ["", f"bench.py's own line in that run: {rec['ms_per_step']:.3f} ms per step, {rec['value']:.0f} seqs/s. "
              f"Dominant class `{dom}`: {rl['avg_launch_us']:.1f} µs per launch by bench.py's live HIP events "
              f"({rl['launches']} sampled launches, every {rl.get('timing_stride', 1)}th) vs "
              + (f"{prof_us:.1f} µs" if prof_us else "n/a") + " (rocprofv3: the class's kernels' total time / its launches); "
              f"{rl['per_launch_flop'] / 1e9:.1f} GFLOP per launch -> {rl['achieved']:.0f} {rl['unit']} = "
              f"{100 * rl['frac']:.1f}% of the {rl['peak']:.0f} {rl['unit']} dense bf16 peak."]
    if plain_json:
        p = json.loads([x for x in open(plain_json) if x.startswith("{")][-1])
        pr = p["roofline"]
        lines += ["", "Under --kernel-trace the events around a class's launches also take in the tracer's "
                  "work per dispatch. The same bench.py without the profiler on the same box "
                  f"(`python bench.py`): {p['ms_per_step']:.3f} ms per step, {p['value']:.0f} seqs/s, "
                  f"`{pr['kernel']}` {pr['avg_launch_us']:.1f} µs per launch by its HIP events "
                  f"-> {pr['achieved']:.0f} {pr['unit']} = {100 * pr['frac']:.1f}% of peak."]
    with open(TRACE_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {TRACE_PROFILE}")


SELECT_PROFILE = os.path.join(ROOT, "profiles", "select_large_n.md")
_SELECT_STAGES = ["init", "count 11b", "reduce", "count 11b", "reduce", "count 10b", "reduce", "scatter", "final"]


def summarize_select(sweep_json, trace_csv, command):
    """Write the large-n select summary: bench.py --select-sweep's line plus per-kernel medians
    from a rocprofv3 kernel trace of the same command (each call is 9 launches in order)."""
    import csv
    import statistics
    rows = json.loads(open(sweep_json).read().strip().splitlines()[-1])["select_sweep"]
    with open(trace_csv) as f:
        tr = sorted((r for r in csv.DictReader(f) if "select_" in r["Kernel_Name"]),
                    key=lambda r: int(r["Start_Timestamp"]))
    nk = len(_SELECT_STAGES)
    calls = [tr[i:i + nk] for i in range(0, len(tr), nk)]
    per_cfg = len(calls) // len(rows)
    lines = ["# ISRTF select above 8192 jobs: device-wide radix selection, n = 2^20 .. 2^24", "",
             "Commands (MI355X, repo root as working tree):", "",
             "    python bench.py --select-sweep", f"    {command}", "",
             "Predictions 250 + 100 * N(0, 0.55^2) (the predictor's output scale), arrivals a random "
             "permutation. `mandatory` = 12 n bytes in (pred + arrival) + 4 k out; HBM fraction = "
             "mandatory bytes / time / 8 TB/s. The implementation reads pred four times (16 n bytes) "
             "and arrivals only for jobs tied on the prediction.", "",
             "| n | k | µs per call (HIP events) | GB/s of mandatory bytes | HBM fraction |",
             "|---:|---:|---:|---:|---:|"]
    for r in rows:
        lines.append(f"| 2^{r['n'].bit_length() - 1} | {r['k']} | {r['us']:.1f} | {r['gbs']:.0f} | {r['hbm_frac']:.3f} |")
    lines += ["", "Per-kernel medians from the trace (µs; a stage that finds its bucket already resolved "
              "returns at once):", "",
              "| n | k | " + " | ".join(_SELECT_STAGES) + " |", "|---:|---:|" + "---:|" * nk]
    for ci, r in enumerate(rows):
        cs = calls[ci * per_cfg + 3:(ci + 1) * per_cfg]
        med = [statistics.median((int(c[j]["End_Timestamp"]) - int(c[j]["Start_Timestamp"])) / 1e3 for c in cs)
               for j in range(nk)]
        lines.append(f"| 2^{r['n'].bit_length() - 1} | {r['k']} | " + " | ".join(f"{v:.1f}" for v in med) + " |")
    lines += ["", "Small launches cost 2-5 µs each (nine per call), so below 2^22 jobs the call is "
              "launch-bound; at k = 8192 the one-work-group bitonic sort of the chosen jobs (~170 µs) "
              "dominates."]
    with open(SELECT_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {SELECT_PROFILE}")


ROUNDS_PROFILE = os.path.join(ROOT, "profiles", "isrtf_rounds_bert_base.md")


def summarize_rounds(rounds_json):
    """Write the ISRTF round-latency summary from bench.py --isrtf-rounds' line."""
    rec = json.loads(open(rounds_json).read().strip().splitlines()[-1])["isrtf_rounds"]
    lines = [f"# ISRTF scheduling rounds: device-resident job table vs host packing", "",
             "Command (MI355X, repo root as working tree):", "", "    python bench.py --isrtf-rounds", "",
             f"{rec['workload']}; the whole stream, every round timed on the host from the start of the "
             "re-score to the chosen jobs on the host. Re-scored jobs per round: the Job Pool (new arrivals "
             "and the jobs that ran in the last window; `pool`) or every in-flight job (`all`). The two drivers "
             f"produce the same schedule (`same_schedule`: {rec['same_schedule']}), and so do the two re-score "
             f"sets (`same_schedule_rescore_all`: {rec.get('same_schedule_rescore_all')}): an unchanged input "
             "gets a bit-identical key.", "",
             "| driver | re-scored | rounds | p50 ms | p99 ms | mean ms | mean re-scored jobs | host-to-device "
             "bytes / round | device-to-host bytes / round |", "|---|---|---:|---:|---:|---:|---:|---:|---:|"]
    for k in ("device_table", "device_table_rescore_all", "host_packing"):
        if k not in rec:
            continue
        r = rec[k]
        lines.append(f"| {k} | {r.get('rescore', 'pool')} | {r['rounds']} | {r['p50_ms']:.2f} | {r['p99_ms']:.2f} | "
                     f"{r['mean_ms']:.2f} | {r['mean_rescored']:.1f} | {r['h2d_bytes_per_round']:,.0f} | "
                     f"{r['d2h_bytes_per_round']:,.0f} |")
    lines += ["", "The encoder pass over the re-scored jobs is most of every round. With the Job Pool only (about "
              "61 jobs, ~22K tokens per round) the two drivers differ by well under a millisecond; the table "
              "moves a fifth of the bytes and synchronises once per round (the chosen slots) instead of twice. "
              "Re-scoring every in-flight job encodes the waiting jobs as well, whose inputs have not changed, "
              "so its rounds cost more for the same schedule."]
    with open(ROUNDS_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {ROUNDS_PROFILE}")


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


def select_sweep(ks=(64, 8192), iters=20):
    """Device-wide ISRTF select at n = 2^20 .. 2^24: time per call and its HBM fraction.

    Predictions are drawn like the predictor's outputs (250 + 100 * N(0, 0.55^2)),
    arrivals are a random permutation. Mandatory bytes = 12 n in (pred + arrival)
    + 4 k out; the implementation reads pred four times (16 n) and arrivals for ties only."""
    import numpy as np
    import torch

    from paper_2505_09142_amd import _elis as E
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream().cuda_stream
    rows = []
    for lg in range(20, 25):
        n = 1 << lg
        rng = np.random.default_rng(lg)
        pred = torch.from_numpy((250.0 + 100.0 * 0.55 * rng.standard_normal(n)).astype(np.float32)).to(dev)
        arr = torch.from_numpy(rng.permutation(n).astype(np.int64)).to(dev)
        wsb = E.elis_select_workspace_bytes(n)
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
        for k in ks:
            idx = torch.empty(k, dtype=torch.int32, device=dev)
            cnt = torch.empty(1, dtype=torch.int32, device=dev)

            def call():
                E.check(E.elis_isrtf_select(pred.data_ptr(), arr.data_ptr(), n, k, idx.data_ptr(), cnt.data_ptr(),
                                            ws.data_ptr(), wsb, stream), "select")
            for _ in range(3):
                call()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(iters):
                call()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / iters * 1e3
            mand = 12.0 * n + 4.0 * k
            rows.append({"n": n, "k": k, "us": us, "mandatory_bytes": mand,
                         "gbs": mand / us / 1e3, "hbm_frac": mand / us / 1e3 / PEAK_HBM_GBS,
                         "read_bytes": 16.0 * n})
            print(f"select n=2^{lg} k={k}: {us:.1f} us, {mand / us / 1e3:.0f} GB/s of mandatory bytes", file=sys.stderr,
                  flush=True)
    st, bits = E.elis_read_status(ws.data_ptr(), stream)
    if st != E.ELIS_OK:
        raise SystemExit(f"device status {st} bits {bits}")
    print(json.dumps({"select_sweep": rows}), flush=True)


GEMM_PLAN_SHAPES = (  # (name, N, K, public epilogue): the encoder products of BERT-base and XLM-R-large
    ("bert_qkv", 2304, 768, 0), ("bert_ffn1", 3072, 768, 1), ("bert_o", 768, 768, 2), ("bert_ffn2", 768, 3072, 2),
    ("xlmr_qkv", 3072, 1024, 0), ("xlmr_ffn1", 4096, 1024, 1), ("xlmr_o", 1024, 1024, 2), ("xlmr_ffn2", 1024, 4096, 2))
GEMM_PLAN_MS = (1024, 2560, 4096, 6144, 8192, 10240, 12288, 14336, 16384, 18432, 20480, 22528, 23931, 26624, 28672,
                30720, 32768, 47000, 92000)
GEMM_PLAN_PROFILE = os.path.join(ROOT, "profiles", "gemm_launch_plans.md")


def gemm_plans(reps=8):
    """Every launch plan the library can choose from, timed one by one (elis_linear_with_plan),
    next to the plan it does choose (elis_linear_plan), over the encoder products of BERT-base
    and XLM-R-large at token counts 1K .. 92K. fp32-out products use the plain residual."""
    import torch

    from paper_2505_09142_amd import _elis as E
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    stream = torch.cuda.current_stream().cuda_stream
    g = torch.Generator(device="cpu").manual_seed(0)
    mmax = max(GEMM_PLAN_MS)
    out = []
    for name, n, k, epi in GEMM_PLAN_SHAPES:
        f32 = epi == 2
        x = (torch.randn(mmax, k, generator=g) * 0.5).to(torch.bfloat16).to(dev)
        w = (torch.randn(n, k, generator=g) * 0.03).to(torch.bfloat16).to(dev)
        bias = torch.zeros(n, device=dev)
        res = torch.randn(mmax, n, device=dev) if f32 else None
        o = torch.empty(mmax, n, device=dev, dtype=torch.float32 if f32 else torch.bfloat16)
        tiles = [t for t in ((256, 256, 1), (128, 128, 2), (64, 128, 2), (64, 128, 1), (64, 64, 4), (64, 64, 2))
                 if n % t[1] == 0]
        for m in GEMM_PLAN_MS:
            plans = []
            for t in tiles:
                plans.append(t + (m, 0, 0, 0))
                per_row, slots = n // t[1], t[2] * cus
                m1 = (-(-m // t[0]) * per_row) // slots * slots // per_row * t[0]
                if 0 < m1 < m:
                    plans += [t + (m1,) + r for r in tiles if r != t]

            def run(plan):
                E.check(E.elis_linear_with_plan(x.data_ptr(), w.data_ptr(), bias.data_ptr(),
                                                res.data_ptr() if f32 else None, m, n, k, epi, plan, o.data_ptr(),
                                                stream), f"{name} {plan}")
            times = {}
            for order in (plans, plans[::-1]):  # two passes in opposite orders, the faster one kept
                for plan in order:
                    for _ in range(2):
                        run(plan)
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    for _ in range(reps):
                        run(plan)
                    e1.record()
                    torch.cuda.synchronize()
                    us = e0.elapsed_time(e1) / reps * 1e3
                    times[plan] = min(us, times.get(plan, us))
            st, chosen = E.elis_linear_plan(m, n, k, epi)
            E.check(st, "elis_linear_plan")
            out.append({"shape": name, "n": n, "k": k, "epi": epi, "m": m, "chosen": list(chosen),
                        "plans": [[list(p), t] for p, t in times.items()]})
            best = min(times, key=times.get)
            print(f"{name} m={m}: chosen {chosen} {times[tuple(chosen)]:.1f} us, fastest {best} {times[best]:.1f} us",
                  file=sys.stderr, flush=True)
        del x, w, res, o
    print(json.dumps({"gemm_plans": out, "cus": cus}), flush=True)


VENDOR_GEMM_MS = (2560, 23931, 92000)
VENDOR_GEMM_PROFILE = os.path.join(ROOT, "profiles", "gemm_vs_hipblaslt.md")


def vendor_gemm(reps=20):
    """The encoder products through elis_linear (the library's own plan and epilogue) next to
    torch's bf16 linear on the same device (hipBLASLt), for reference: the same product with its
    bias in bf16 (like for like), and for the GELU and residual products the library's fused
    epilogue against the vendor product plus torch's separate GELU / residual add."""
    import torch
    import torch.nn.functional as F

    from paper_2505_09142_amd import _elis as E
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream().cuda_stream
    g = torch.Generator(device="cpu").manual_seed(0)
    mmax = max(VENDOR_GEMM_MS)

    def timed(fn):
        best = None
        for _ in range(2):  # two passes, the faster kept
            for _ in range(3):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / reps * 1e3
            best = us if best is None else min(best, us)
        return best

    rows = []
    for name, n, k, epi in GEMM_PLAN_SHAPES:
        x = (torch.randn(mmax, k, generator=g) * 0.5).to(torch.bfloat16).to(dev)
        w = (torch.randn(n, k, generator=g) * 0.03).to(torch.bfloat16).to(dev)
        bias = (torch.randn(n, generator=g) * 0.1).to(dev)
        bias16 = bias.to(torch.bfloat16)
        res = torch.randn(mmax, n, device=dev) if epi == 2 else None
        ob = torch.empty(mmax, n, device=dev, dtype=torch.bfloat16)
        of = torch.empty(mmax, n, device=dev, dtype=torch.float32) if epi == 2 else None
        for m in VENDOR_GEMM_MS:
            xm = x[:m]

            def ours(e):
                o = of if e == 2 else ob
                E.check(E.elis_linear(xm.data_ptr(), w.data_ptr(), bias.data_ptr(),
                                      res.data_ptr() if e == 2 else None, m, n, k, e, o.data_ptr(), stream), name)

            r = {"shape": name, "m": m, "n": n, "k": k, "epi": epi, "flop": 2.0 * m * n * k,
                 "ours_bias_us": timed(lambda: ours(0)),
                 "vendor_bias_us": timed(lambda: F.linear(xm, w, bias16))}
            if epi == 1:
                r["ours_epi_us"] = timed(lambda: ours(1))
                r["vendor_epi_us"] = timed(lambda: F.gelu(F.linear(xm, w, bias16)))
            elif epi == 2:
                rm = res[:m]
                r["ours_epi_us"] = timed(lambda: ours(2))
                r["vendor_epi_us"] = timed(lambda: torch.add(rm, F.linear(xm, w, bias16)))
            rows.append(r)
            print(f"{name} m={m}: ours {r['ours_bias_us']:.1f} us, vendor {r['vendor_bias_us']:.1f} us",
                  file=sys.stderr, flush=True)
        del x, w, res, ob, of
    print(json.dumps({"vendor_gemm": rows, "device": torch.cuda.get_device_name(0),
                      "torch": torch.__version__}), flush=True)


def summarize_vendor_gemm(js, command):
    d = json.loads([x for x in open(js) if x.startswith("{")][-1])
    rows = d["vendor_gemm"]
    tf = lambda r, key: r["flop"] / (r[key] * 1e-6) / 1e12
    lines = ["# Encoder GEMMs: this library vs torch's bf16 linear (hipBLASLt), same device", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             f"torch {d['torch']} on {d['device']}. Each product is timed as the best of two passes of 20 "
             "back-to-back calls (HIP events, inputs resident). `bias` columns: the same product and bias, "
             "bf16 out (this library: `elis_linear` with the bf16 bias epilogue and its own launch plan; "
             "vendor: `F.linear`). `fused` columns: the product as the encoder runs it, this library's "
             "fused epilogue (GELU, or fp32 out plus the residual) against `F.linear` followed by "
             "torch's `F.gelu` or residual add. TFLOP/s counts 2·M·N·K; % is of the 2500 TFLOP/s dense "
             "bf16 peak.", "",
             "| shape | M | N | K | bias: ours µs | vendor µs | ours / vendor speed | ours % peak | "
             "vendor % peak | fused: ours µs | vendor µs | speed-up |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for r in rows:
        fused = (f"{r['ours_epi_us']:.1f} | {r['vendor_epi_us']:.1f} | {r['vendor_epi_us'] / r['ours_epi_us']:.2f}×"
                 if "ours_epi_us" in r else "- | - | -")
        lines.append(f"| {r['shape']} | {r['m']:,} | {r['n']} | {r['k']} | {r['ours_bias_us']:.1f} | "
                     f"{r['vendor_bias_us']:.1f} | {r['vendor_bias_us'] / r['ours_bias_us']:.2f}× | "
                     f"{100 * tf(r, 'ours_bias_us') / PEAK_BF16_TFLOPS:.1f} | "
                     f"{100 * tf(r, 'vendor_bias_us') / PEAK_BF16_TFLOPS:.1f} | {fused} |")
    tot_o = sum(r["ours_bias_us"] for r in rows)
    tot_v = sum(r["vendor_bias_us"] for r in rows)
    lines += ["", f"Summed over all rows (bias epilogue): this library {tot_o:,.0f} µs, vendor {tot_v:,.0f} µs "
              f"({tot_v / tot_o:.2f}×)."]
    fo = [r for r in rows if "ours_epi_us" in r]
    if fo:
        a, b = sum(r["ours_epi_us"] for r in fo), sum(r["vendor_epi_us"] for r in fo)
        lines.append(f"Fused products (GELU and residual rows): this library {a:,.0f} µs, vendor + torch "
                     f"{b:,.0f} µs ({b / a:.2f}×).")
    with open(VENDOR_GEMM_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {VENDOR_GEMM_PROFILE}")


def summarize_gemm_plans(js, command):
    rec = json.loads([x for x in open(js) if x.startswith("{")][-1])
    rows = rec["gemm_plans"]

    def tile(p):
        return f"{p[0]}×{p[1]}/{p[2]}"

    def label(p):
        return tile(p) if p[4] == 0 else f"{tile(p)} + {tile(p[4:7])} from row {p[3]:,}"
    lines = ["# GEMM launch plans: every plan timed vs the one the library picks", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             "For each encoder product of BERT-base and XLM-R-large (fp32-out products with the plain residual) "
             "and each token count M, every plan the library can choose from is timed through "
             "`elis_linear_with_plan`: one launch of tiles (written rows×columns/work-groups per CU: 256×256/1, "
             "128×128/2, 64×128/2, 64×128/1 with 4 stages, 64×64/4, 64×64/2 with 4 stages), or large tiles over "
             "the rows that fill whole rounds plus a second launch of another "
             "configuration over the rest. `chosen` is `elis_linear_plan`'s pick (the launch-time model); "
             "`fastest` the best measured; the fixed columns are what one configuration alone takes.", "",
             "| shape | chosen / fastest, summed over M | 256×256 alone | 128×128 alone |", "|---|---:|---:|---:|"]
    tot = {"chosen": 0.0, "fastest": 0.0}
    by_shape = {}
    for r in rows:
        t = {tuple(p): us for p, us in r["plans"]}
        m = r["m"]
        c = t[tuple(r["chosen"])]
        f = min(t.values())
        s = by_shape.setdefault(r["shape"], {"chosen": 0.0, "fastest": 0.0, "256": 0.0, "128": 0.0, "has256": True})
        s["chosen"] += c
        s["fastest"] += f
        s["128"] += t[(128, 128, 2, m, 0, 0, 0)]
        if (256, 256, 1, m, 0, 0, 0) in t:
            s["256"] += t[(256, 256, 1, m, 0, 0, 0)]
        else:
            s["has256"] = False
        tot["chosen"] += c
        tot["fastest"] += f
    for name, s in by_shape.items():
        lines.append(f"| {name} | {s['chosen'] / s['fastest']:.3f} | "
                     + (f"{s['256'] / s['fastest']:.3f}" if s["has256"] else "-") + f" | {s['128'] / s['fastest']:.3f} |")
    lines += ["", f"All shapes and sizes: the chosen plans take {tot['chosen'] / tot['fastest']:.4f}× the time of the "
              "fastest measured ones.", "",
              "Per size, BERT-base at the benchmark's 23,931 tokens and at a small and a large batch:", "",
              "| shape | M | chosen plan | µs | fastest plan | µs |", "|---|---:|---|---:|---|---:|"]
    for r in rows:
        if r["shape"].startswith("bert") and r["m"] in (2560, 23931, 92000):
            t = {tuple(p): us for p, us in r["plans"]}
            best = min(t, key=t.get)
            lines.append(f"| {r['shape']} | {r['m']:,} | {label(r['chosen'])} | {t[tuple(r['chosen'])]:.1f} | "
                         f"{label(list(best))} | {t[best]:.1f} |")
    with open(GEMM_PLAN_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {GEMM_PLAN_PROFILE}")


def isrtf_rounds(max_rounds=None):
    """Per-round scheduling latency of the ISRTF loop over the 4096-request stream (Poisson
    arrivals at 20/s, 50-token windows, batch cap 64), device-resident job table vs host
    packing. Latency = host wall time from the start of a round's re-score to the chosen
    jobs on the host (append / pack / predict / store / select, or host packing + copies)."""
    import numpy as np
    import torch

    from paper_2505_09142_amd.device import DeviceWeights, Predictor
    from paper_2505_09142_amd.driver import DeviceRoundDriver, HostRoundDriver
    from paper_2505_09142_amd.scheduler import run_isrtf
    from workloads import S_ISRTF, make_requests, make_weights
    s = S_ISRTF
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    W = make_weights(s.shape, s.weight_seed)
    pr = Predictor(DeviceWeights(s.shape, W.device, dev), dev)
    req = make_requests(s)
    out = {"workload": f"ISRTF loop: {len(req.prompt)} requests, Poisson {s.rate_per_s}/s, window {s.window}, "
                       f"batch cap {s.batch_cap}, BERT-base-shaped predictor (max_pos {s.shape.max_pos})"}
    chosen = {}

    def make(name):
        if name.startswith("device_table"):
            return DeviceRoundDriver(pr, 2048, s.shape.max_pos, dev)
        return HostRoundDriver(pr, s.shape.max_pos, len(req.prompt), dev)

    # (row, driver, which jobs are re-scored each round): the Job Pool only (new arrivals and the
    # jobs that ran in the last window), or every in-flight job, as the stream's configuration
    # states it; with a deterministic encoder both give the same keys and so the same schedule.
    for name, rescore in (("device_table", "pool"), ("device_table_rescore_all", "all"),
                          ("host_packing", "pool")):
        # warm-up rounds on the same driver type, then the measured run from the start
        run_isrtf(req.arrival_t, req.prompt, req.response, make(name), window=s.window,
                  step_cost=s.step_cost_s, batch_cap=s.batch_cap, rescore=rescore, max_rounds=10)
        drv = make(name)
        res = run_isrtf(req.arrival_t, req.prompt, req.response, drv, window=s.window, step_cost=s.step_cost_s,
                        batch_cap=s.batch_cap, rescore=rescore, max_rounds=max_rounds)
        lat = np.array([r.latency_s for r in res.rounds]) * 1e3
        n_rescored = np.array([len(r.rescored) for r in res.rounds])
        out[name] = {"rescore": rescore, "rounds": len(res.rounds), "p50_ms": float(np.percentile(lat, 50)),
                     "p99_ms": float(np.percentile(lat, 99)), "mean_ms": float(lat.mean()),
                     "mean_rescored": float(n_rescored.mean()), "max_candidates":
                         int(max(len(r.candidates) for r in res.rounds)),
                     "mean_jct_s": float(np.nanmean(res.jct)),
                     "h2d_bytes_per_round": drv.h2d_bytes / len(res.rounds),
                     "d2h_bytes_per_round": drv.d2h_bytes / len(res.rounds)}
        chosen[name] = [r.chosen for r in res.rounds]
        print(f"{name}: {len(res.rounds)} rounds, p50 {out[name]['p50_ms']:.2f} ms, p99 {out[name]['p99_ms']:.2f} ms",
              file=sys.stderr, flush=True)
    out["same_schedule"] = chosen["device_table"] == chosen["host_packing"]
    out["same_schedule_rescore_all"] = chosen["device_table"] == chosen["device_table_rescore_all"]
    print(json.dumps({"isrtf_rounds": out}), flush=True)


ROUNDS100_PROFILE = os.path.join(ROOT, "profiles", "bert_base_b256_x100_rounds.md")


def rounds_b256():
    """The 100-round workload on the device job table: 256 in-flight sequences (prompt +
    generated-so-far, truncated to 512), each gaining one token per round; every round appends
    the new tokens, packs all 256 inputs on the device, re-predicts them and selects 128. Latency
    per round = host wall time from the append to the chosen slots on the host; GPU time per
    round = HIP events around append + pack + predict + select on the stream."""
    import numpy as np
    import torch

    from paper_2505_09142_amd.device import DeviceWeights, Predictor
    from paper_2505_09142_amd.driver import DeviceRoundDriver
    from workloads import W_BERT_B256_ROUNDS as w, make_weights
    from workloads.gen import RoundStream
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    W = make_weights(w.shape, w.weight_seed)
    pr = Predictor(DeviceWeights(w.shape, W.device, dev), dev)
    rs = RoundStream(w)
    n = w.n_seqs
    base = (rs.prompt + rs.gen0).astype(np.int64)
    prompts = [st[:int(b)] for st, b in zip(rs.streams, base)]
    responses = [st[int(b):] for st, b in zip(rs.streams, base)]
    jobs = list(range(n))

    def run(rounds):
        drv = DeviceRoundDriver(pr, n, w.shape.max_pos, dev)
        drv.start(jobs, rs.arrival)
        gen = np.zeros(n, dtype=np.int64)
        wall, gpu, toks = [], [], []
        for r in range(rounds):
            gen[:] = r
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0 = time.perf_counter()
            e0.record()
            drv.sync_tokens(jobs, prompts, responses, gen)
            drv.predict(jobs)
            chosen = drv.select(jobs, w.batch_cap)
            e1.record()
            wall.append(time.perf_counter() - t0)
            torch.cuda.synchronize()
            gpu.append(e0.elapsed_time(e1) * 1e-3)
            toks.append(int(np.minimum(base + r, w.shape.max_pos).sum()))
            assert len(chosen) == w.batch_cap
        st, bits = drv.table.status()
        if st != 0:
            raise SystemExit(f"job table status {st} bits {bits}")
        return np.array(wall), np.array(gpu), np.array(toks)

    run(3)  # warm-up
    wall, gpu, toks = run(w.rounds)
    out = {"workload": f"{w.name}: {n} in-flight sequences, BERT-base-shaped predictor, +1 token per round, "
                       f"select {w.batch_cap}, {w.rounds} rounds on the device job table",
           "rounds": int(w.rounds), "tokens_round0": int(toks[0]), "tokens_round_last": int(toks[-1]),
           "p50_ms": float(np.percentile(wall, 50) * 1e3), "p99_ms": float(np.percentile(wall, 99) * 1e3),
           "gpu_p50_ms": float(np.percentile(gpu, 50) * 1e3), "gpu_mean_ms": float(gpu.mean() * 1e3),
           "seqs_per_s": float(n * len(gpu) / gpu.sum()), "tokens_per_s": float(toks.sum() / gpu.sum()),
           "gpu_ms_round0": float(gpu[0] * 1e3), "gpu_ms_round_last": float(gpu[-1] * 1e3)}
    print(json.dumps({"rounds_b256": out}), flush=True)


def summarize_rounds100(js, command):
    rec = json.loads(open(js).read().strip().splitlines()[-1])["rounds_b256"]
    lines = ["# 100 scheduling rounds at 256 in-flight sequences (BERT-base-shaped predictor)", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             f"{rec['workload']}. Every round appends each sequence's new token to the device job table, packs "
             "all 256 inputs on the device (first token plus the most recent 511 past 512), re-predicts every one "
             "and selects 128; one host synchronisation per round (the chosen slots).", "",
             "| rounds | tokens (round 0 → last) | GPU ms / round (p50, mean) | GPU ms round 0 → last | host wall ms / round (p50, p99) | seqs/s | tokens/s |",
             "|---:|---|---|---|---|---:|---:|",
             f"| {rec['rounds']} | {rec['tokens_round0']:,} → {rec['tokens_round_last']:,} | {rec['gpu_p50_ms']:.2f}, "
             f"{rec['gpu_mean_ms']:.2f} | {rec['gpu_ms_round0']:.2f} → {rec['gpu_ms_round_last']:.2f} | "
             f"{rec['p50_ms']:.2f}, {rec['p99_ms']:.2f} | {rec['seqs_per_s']:,.0f} | {rec['tokens_per_s']:,.0f} |"]
    with open(ROUNDS100_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {ROUNDS100_PROFILE}")


WORKLOADS_PROFILE = os.path.join(ROOT, "profiles", "workloads_summary.md")


def summarize_workloads(paths, command):
    """One table over bench.py lines of several --workload runs."""
    lines = ["# Predict + select per workload (one MI355X)", "",
             "Command (MI355X, repo root as working tree), once per workload:", "", f"    {command}", "",
             "One step = elis_predict_remaining + elis_isrtf_select on a batch resident in HBM; GEMM and attention "
             "MFMA utilisation = algorithmic FLOPs / per-class kernel time / 2.5 PFLOP/s (HIP events around each "
             "launch); the roofline column is bench.py's dominant kernel class.", "",
             "| workload | sequences | tokens | ms / step (p50) | seqs/s | tokens/s | GEMM MFMA util | attention MFMA util | dominant kernel (frac of peak) |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---|"]
    for pth in paths:
        d = json.loads([x for x in open(pth) if x.startswith("{")][-1])
        c, rf = d["config"], d["roofline"]
        name = c["workload"].split(":")[0]
        lines.append(f"| {name} | {c['n_seqs']} | {c['total_tokens']:,} | {d['p50_ms']:.3f} | {d['value']:,.0f} | "
                     f"{d['tokens_per_s']:,.0f} | {d['mfma_util_gemm']:.3f} | {d['mfma_util_attention']:.3f} | "
                     f"{rf['kernel']} ({rf['frac']:.3f}) |")
    with open(WORKLOADS_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {WORKLOADS_PROFILE}")


POLICY_PROFILE = os.path.join(ROOT, "profiles", "policy_study.md")


def policy_study():
    """Synthetic analogue of the paper's scheduler comparison (Fig. 5 and 6): FCFS, ISRTF and SJF
    on the device job table (keys cached in HBM, selection by elis_jobs_select[_aged]), 200
    requests with Gamma(0.73) intervals, batch caps 1/2/4 at 1x/3x/5x the average request rate,
    3 shuffled repetitions each. ISRTF's keys come from a stand-in predictor with the paper's
    final MAE (true remaining + Laplace noise); starvation control (aging) and re-prefill cost
    are measured at batch 4; one ISRTF run per rate uses the BERT-base-shaped encoder on the GPU
    (random weights: its predictions carry no length information)."""
    import numpy as np
    import torch

    from paper_2505_09142_amd.device import DeviceWeights, Predictor
    from paper_2505_09142_amd.driver import DeviceRoundDriver
    from paper_2505_09142_amd.scheduler import run_schedule
    from workloads import BERT_BASE, POLICY_STUDY, accuracy_model_keys, make_policy_requests, make_weights
    st = POLICY_STUDY
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    runs = []

    def one(policy, cap, rps, rep, aging=0.0, prefill=0.0, encoder=None):
        req = make_policy_requests(st, cap, rps, rep)
        rem = np.array([len(r) for r in req.response])

        def key_fn(jobs, gen):
            jobs = np.asarray(jobs)
            return accuracy_model_keys(st.data_seed, jobs, gen[jobs], rem[jobs] - gen[jobs], st.accuracy_mae)
        drv = DeviceRoundDriver(encoder, 256, BERT_BASE.max_pos, dev)
        res = run_schedule(req.arrival_t, req.prompt, req.response, drv, window=st.window,
                           step_cost=st.step_cost_s, batch_cap=cap, policy=policy,
                           key_fn=key_fn if (policy == "isrtf" and encoder is None) else None,
                           aging=aging, prefill_cost=prefill)
        lat = np.array([r.latency_s for r in res.rounds]) * 1e3
        name = policy + ("_encoder" if encoder is not None else "") + (f"_aging{aging:g}" if aging else "") + \
            (f"_prefill{prefill:g}" if prefill else "")
        runs.append({"variant": name, "batch_cap": cap, "rps_multiple": rps, "repetition": rep,
                     "mean_jct_s": float(res.jct.mean()), "mean_queue_s": float(res.queue_delay.mean()),
                     "p99_jct_s": float(np.percentile(res.jct, 99)), "max_jct_s": float(res.jct.max()),
                     "preemptions": int(res.preemptions.sum()), "rounds": len(res.rounds),
                     "round_p50_ms": float(np.median(lat))})
        t, bits = drv.table.status()
        if t != 0:
            raise SystemExit(f"job table status {t} bits {bits}")

    for cap in st.batch_caps:
        for rps in st.rps_multiples:
            for rep in range(st.repetitions):
                for policy in ("fcfs", "isrtf", "sjf"):
                    one(policy, cap, rps, rep)
                if cap == max(st.batch_caps):
                    one("isrtf", cap, rps, rep, aging=st.aging)
                    one("isrtf", cap, rps, rep, prefill=st.prefill_cost_s)
                    one("isrtf", cap, rps, rep, aging=st.aging, prefill=st.prefill_cost_s)
            print(f"policy study: batch {cap}, {rps:g}x done", file=sys.stderr, flush=True)
    W = make_weights(BERT_BASE, 1002)
    pr = Predictor(DeviceWeights(BERT_BASE, W.device, dev), dev)
    cap = max(st.batch_caps)
    for rps in st.rps_multiples:
        one("isrtf", cap, rps, 0, encoder=pr)
    print("policy study: encoder runs done", file=sys.stderr, flush=True)
    print(json.dumps({"policy_study": {"requests": st.n_requests, "window": st.window,
                                       "step_cost_s": st.step_cost_s, "gamma_shape": st.gamma_shape,
                                       "accuracy_mae": st.accuracy_mae, "aging": st.aging,
                                       "prefill_cost_s": st.prefill_cost_s, "runs": runs}}), flush=True)


def summarize_policy(study_json, command):
    """Write the policy-study summary (mean over repetitions) from bench.py --policy-study's line."""
    import collections
    rec = json.loads(open(study_json).read().strip().splitlines()[-1])["policy_study"]
    agg = collections.defaultdict(list)
    for r in rec["runs"]:
        agg[(r["variant"], r["batch_cap"], r["rps_multiple"])].append(r)
    mean = {k: {f: sum(x[f] for x in v) / len(v) for f in ("mean_jct_s", "mean_queue_s", "p99_jct_s",
                                                          "preemptions", "rounds", "round_p50_ms")}
            for k, v in agg.items()}
    variants = sorted({k[0] for k in mean}, key=lambda v: (v != "fcfs", v != "isrtf", v != "sjf", v))
    caps = sorted({k[1] for k in mean})
    rpss = sorted({k[2] for k in mean})
    lines = ["# Scheduler policy study (synthetic analogue of Fig. 5 and 6)", "",
             "Command (MI355X, repo root as working tree):", "", f"    {command}", "",
             f"{rec['requests']} synthetic requests per run (prompt lognormal(200, 0.8), response lognormal(250, 1.0) "
             f"capped at 2048), Gamma(shape {rec['gamma_shape']}) request intervals at k x batch / (mean response "
             f"length x {rec['step_cost_s'] * 1e3:g} ms per decode step) requests/s, {rec['window']}-token windows, "
             "the same request set shuffled for each of 3 repetitions (means below). Every run is the scheduling "
             "loop on the device job table: keys cached in HBM, batches chosen by `elis_jobs_select` / "
             "`elis_jobs_select_aged`; the same trajectories are reproduced exactly by the oracle simulator in "
             "`tests/test_gpu_policies.py`.", "",
             f"ISRTF keys: a stand-in predictor with the paper's final MAE ({rec['accuracy_mae']} tokens): true "
             "remaining length + Laplace noise. `isrtf_encoder`: the BERT-base-shaped encoder on the GPU with random "
             "weights (no length information, so it ranks jobs arbitrarily). Aging: "
             f"{rec['aging']:g} tokens per second of waiting; re-prefill cost {rec['prefill_cost_s'] * 1e3:g} ms "
             "per token for a preempted job that resumes.", "",
             "## Mean JCT (s) and improvement over FCFS", "",
             "| batch | rate | " + " | ".join(variants) + " |", "|---|---|" + "---:|" * len(variants)]
    for cap in caps:
        for rps in rpss:
            base = mean.get(("fcfs", cap, rps))
            cells = []
            for v in variants:
                m = mean.get((v, cap, rps))
                if m is None:
                    cells.append("")
                elif v == "fcfs" or base is None:
                    cells.append(f"{m['mean_jct_s']:.2f}")
                else:
                    cells.append(f"{m['mean_jct_s']:.2f} ({100 * (1 - m['mean_jct_s'] / base['mean_jct_s']):+.1f}%)")
            lines.append(f"| {cap} | {rps:g}x | " + " | ".join(cells) + " |")
    lines += ["", "## Mean queuing delay (s), preemptions per run, scheduling rounds per run", "",
              "| variant | batch | rate | queuing delay | p99 JCT | preemptions | rounds | p50 round ms |",
              "|---|---|---|---:|---:|---:|---:|---:|"]
    for v in variants:
        for cap in caps:
            for rps in rpss:
                m = mean.get((v, cap, rps))
                if m is None:
                    continue
                lines.append(f"| {v} | {cap} | {rps:g}x | {m['mean_queue_s']:.2f} | {m['p99_jct_s']:.2f} | "
                             f"{m['preemptions']:.0f} | {m['rounds']:.0f} | {m['round_p50_ms']:.3f} |")
    lines += ["", "Round latency: host wall time of one round's key update plus selection on the device, "
              "including the host-to-device upload of the candidates and the read-back of the chosen jobs "
              "(the encoder variant includes the predictor pass)."]
    with open(POLICY_PROFILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {POLICY_PROFILE}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="bert_base_b64")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-b256-round0", action="store_true",
                    help="leave out the batch-256 round-0 passes that follow the steps (profiler runs of "
                         "the batch-64 workload, so only its dispatches are counted)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run a plain device copy of this many MiB three times before the steps "
                         "(reference dispatches for PMC byte counters)")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the HBM-traffic summary from two rocprofv3 --pmc counter_collection.csv files")
    ap.add_argument("--summarize-rounds", metavar="ROUNDS_JSON",
                    help="write the ISRTF round-latency summary")
    ap.add_argument("--isrtf-rounds", action="store_true",
                    help="per-round latency of the ISRTF loop: device job table vs host packing")
    ap.add_argument("--rounds-b256", action="store_true",
                    help="the 100-round, 256-sequence workload on the device job table (per-round latency)")
    ap.add_argument("--summarize-rounds-b256", nargs=2, metavar=("JSON", "COMMAND"),
                    help="write the 100-round summary")
    ap.add_argument("--summarize-workloads", nargs="+", metavar="BENCH_JSON",
                    help="write the per-workload summary from several bench.py lines (last arg: the command)")
    ap.add_argument("--policy-study", action="store_true",
                    help="FCFS / ISRTF / SJF, aging and re-prefill cost on the device job table (Fig. 5/6 analogue)")
    ap.add_argument("--summarize-policy", nargs=2, metavar=("STUDY_JSON", "COMMAND"),
                    help="write the policy-study summary")
    ap.add_argument("--gemm-plans", action="store_true",
                    help="time every GEMM launch plan against the library's choice (encoder products, M = 1K .. 92K)")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="time the encoder GEMMs against torch's bf16 linear (hipBLASLt) on the same device")
    ap.add_argument("--summarize-vendor-gemm", nargs=2, metavar=("JSON", "COMMAND"),
                    help="write the GEMM-vs-vendor summary")
    ap.add_argument("--summarize-gemm-plans", nargs=2, metavar=("JSON", "COMMAND"),
                    help="write the GEMM launch-plan summary")
    ap.add_argument("--select-sweep", action="store_true",
                    help="time the device-wide select at n = 2^20 .. 2^24 instead of the step")
    ap.add_argument("--summarize-select", nargs=3, metavar=("SWEEP_JSON", "TRACE_CSV", "COMMAND"),
                    help="write the large-n select summary")
    ap.add_argument("--summarize-trace", nargs="+", metavar="ARG",
                    help="write the kernel-trace summary from a rocprofv3 kernel_stats.csv: "
                         "STATS_CSV BENCH_JSON COMMAND [PLAIN_BENCH_JSON]")
    ap.add_argument("--summarize-issue", nargs=2, metavar=("PMC_CSV", "COMMAND"),
                    help="write the instruction-mix / LDS-conflict summary from a --pmc pass of ISSUE_COUNTERS")
    ap.add_argument("--summarize-mfma", nargs=3, metavar=("PMC_CSV", "BENCH_JSON", "COMMAND"),
                    help="write the MFMA-busy summary from a SQ_VALU_MFMA_BUSY_CYCLES / SQ_BUSY_CYCLES pass")
    ap.add_argument("--pmc-command", action="append", default=[],
                    help="with --summarize-pmc: the command of each pass, recorded in the summary")
    args = ap.parse_args()
    if args.summarize_rounds:
        summarize_rounds(args.summarize_rounds)
        return
    if args.isrtf_rounds:
        isrtf_rounds()
        return
    if args.rounds_b256:
        rounds_b256()
        return
    if args.summarize_rounds_b256:
        summarize_rounds100(*args.summarize_rounds_b256)
        return
    if args.summarize_workloads:
        summarize_workloads(args.summarize_workloads[:-1], args.summarize_workloads[-1])
        return
    if args.policy_study:
        policy_study()
        return
    if args.summarize_policy:
        summarize_policy(*args.summarize_policy)
        return
    if args.summarize_select:
        summarize_select(*args.summarize_select)
        return
    if args.select_sweep:
        select_sweep()
        return
    if args.gemm_plans:
        gemm_plans()
        return
    if args.vendor_gemm:
        vendor_gemm()
        return
    if args.summarize_vendor_gemm:
        summarize_vendor_gemm(*args.summarize_vendor_gemm)
        return
    if args.summarize_gemm_plans:
        summarize_gemm_plans(*args.summarize_gemm_plans)
        return
    if args.summarize_trace:
        a = args.summarize_trace  # STATS_CSV BENCH_JSON COMMAND [PLAIN_BENCH_JSON]
        if len(a) not in (3, 4):
            ap.error("--summarize-trace takes STATS_CSV BENCH_JSON COMMAND [PLAIN_BENCH_JSON]")
        summarize_trace(a[0], a[2], a[1], a[3] if len(a) == 4 else None)
        return
    if args.summarize_issue:
        summarize_issue(*args.summarize_issue)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.copy_calibration_mib, args.workload, args.pmc_command)
        return
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

    if args.copy_calibration_mib:
        src = torch.ones(args.copy_calibration_mib * 2 ** 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

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
        kind, per, count = alg[name]
        if nl != count * args.steps:
            raise SystemExit(f"{name}: {nl} launches in {args.steps} steps, the work model expects {count} per step")
        per_launch = sum(per) / count
        avg_s = ms / nl * 1e-3
        rate = per_launch / avg_s / (1e12 if kind == "flop" else 1e9)
        kernels[name] = {"launches_per_step": nl / args.steps, "avg_us": avg_s * 1e6, "ms_per_step": ms / args.steps,
                         ("tflops" if kind == "flop" else "gbs"): rate}
    dominant = max(kernels, key=lambda k: kernels[k]["ms_per_step"])

    # Timed region: per-step events, and the dominant class timed on a sample of its launches:
    # every `stride`-th launch, stride coprime to the launches per step so that the sample rotates
    # over the layers. A timed dispatch costs a few microseconds of idle GPU around it, which
    # timing every launch would add to the step time.
    per_step = round(kernels[dominant]["launches_per_step"])
    stride = next(s for s in (13, 17, 19, 23) if per_step % s)
    E.elis_timing_reset()
    E.elis_timing_stride(stride)
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
    E.elis_timing_stride(1)
    _, dl, dms = E.elis_timing_read(E.K[dominant])
    elapsed = t1 - t0
    lat = np.array([a.elapsed_time(c) for a, c in evs])
    st, bits = pr.status()
    if st != E.ELIS_OK:
        raise SystemExit(f"device status {st} bits {bits}")

    kind, per, _ = alg[dominant]
    per_launch = sampled_work(per, stride, dl)   # the work of exactly the launches the sample timed
    avg_s = dms / dl * 1e-3
    if kind == "flop":
        achieved, peak, unit, bound = per_launch / avg_s / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s", "mfma"
    else:
        achieved, peak, unit, bound = per_launch / avg_s / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
    gemm_flop = sum(sum(alg[k][1]) for k in ("gemm_qkv", "gemm_o", "gemm_ffn1", "gemm_ffn2"))
    gemm_s = sum(kernels[k]["ms_per_step"] for k in ("gemm_qkv", "gemm_o", "gemm_ffn1", "gemm_ffn2")) * 1e-3
    att_s = kernels["attention"]["ms_per_step"] * 1e-3
    att_flop = sum(alg["attention"][1])

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
        "config": {"workload": _describe(w),
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
                     "avg_launch_us": avg_s * 1e6, "launches": dl, "timing_stride": stride},
        "kernels": kernels,
    }
    if args.workload == "bert_base_b64" and not args.no_b256_round0:
        out["b256_round0"] = b256_round0(pr)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, W, b, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def b256_round0(pr, passes=5):
    """The batch-256 workload's first round (the same BERT-base predictor weights; 256 sequences,
    ~92K tokens), outside the timed steps: per-class kernel time of a few predictor passes, so the
    GEMM and attention matrix-core utilisation at that size comes with every bench line."""
    import torch
    from paper_2505_09142_amd import _elis as E
    from paper_2505_09142_amd.device import upload_batch
    from workloads import W_BERT_B256_ROUNDS
    from workloads.gen import RoundStream
    w = W_BERT_B256_ROUNDS
    b = RoundStream(w).batch(0)
    ids, cu, arr = upload_batch(b, pr.device)
    pred = torch.empty(b.n, dtype=torch.float32, device=pr.device)
    for _ in range(2):
        pr.predict(ids, cu, b.max_seqlen, out_pred=pred)
    torch.cuda.synchronize()
    alg = _algorithmic(w, b)
    E.elis_timing_reset()
    E.elis_timing_enable((1 << len(E.KERNEL_CLASSES)) - 1)
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    for _ in range(passes):
        pr.predict(ids, cu, b.max_seqlen, out_pred=pred)
    a1.record()
    torch.cuda.synchronize()
    E.elis_timing_enable(0)
    cls_ms = {name: E.elis_timing_read(E.K[name])[2] / passes for name in E.KERNEL_CLASSES}
    E.elis_timing_reset()
    gemm = ("gemm_qkv", "gemm_o", "gemm_ffn1", "gemm_ffn2")
    gemm_flop = sum(sum(alg[k][1]) for k in gemm)
    gemm_ms = sum(cls_ms[k] for k in gemm)
    return {"workload": f"{w.name} round 0: {b.n} sequences, {b.total} tokens, predict only",
            "total_tokens": int(b.total), "ms_per_pass_timed_classes": a0.elapsed_time(a1) / passes,
            "mfma_util_gemm": gemm_flop / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "mfma_util_attention": sum(alg["attention"][1]) / (cls_ms["attention"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "gemm_tflops": {k: sum(alg[k][1]) / (cls_ms[k] * 1e-3) / 1e12 for k in gemm}}


if __name__ == "__main__":
    main()
