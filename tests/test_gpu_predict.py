"""End-to-end parity of elis_predict_remaining + elis_isrtf_select against the
fp64 oracle on the workloads' own seeded inputs.

Bars: predictions within relative 2e-2 (relative to max(|p_oracle|, 1)), the
unshifted head output y = (p - out_shift) / out_scale within 2e-2 of the
batch's largest |y_oracle|, final hidden states within max-abs 5e-2, the
selection bit-exact when both sides see the same fp32 predictions, and end to
end (GPU predictions vs oracle predictions) equal selected sets whenever the
oracle's gap at the cut exceeds twice the largest prediction error. This file
holds the small shapes, evaluated on every sequence, and the GPU-only
invariants; the full-size batches are in test_gpu_full_size.py.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2505_09142_amd import _elis as E
from paper_2505_09142_amd.device import DeviceWeights, Predictor, upload_batch
from tests.gpu_util import dev, note
from tests.parity_log import record
from workloads import (TINY, W_BERT_B64, W_TINY, W_TINY_CLS_LIN8, W_TINY_HEAD8, bf16_bits_to_f32, make_batch,
                       make_weights, pack)

pytestmark = pytest.mark.gpu

PRED_RTOL = 2e-2
HIDDEN_ATOL = 5e-2


_cache = {}


def predictor(shape, seed):
    key = (shape, seed)
    if key not in _cache:
        W = make_weights(shape, seed)
        _cache.clear()
        _cache[key] = (W, Predictor(DeviceWeights(shape, W.device)))
    return _cache[key]


def run(pr, batch, want_hidden=True):
    ids, cu, arr = upload_batch(batch)
    pred, hid = pr.predict(ids, cu, batch.max_seqlen, want_hidden=want_hidden)
    st, bits = pr.status()
    assert st == E.ELIS_OK, (st, bits)
    return pred.cpu().numpy(), (hid.cpu().numpy() if hid is not None else None), arr


def rel_err(p, ref):
    return np.abs(p - ref) / np.maximum(np.abs(ref), 1.0)


Y_RTOL = 2e-2


def y_rel(p, ref, shape):
    """Error of the unshifted head output y = (p - out_shift) / out_scale, relative to the batch's
    largest |y_ref|: the fixed shift of the prediction does not dilute it."""
    y = (np.asarray(p, np.float64) - shape.out_shift) / shape.out_scale
    y_ref = (np.asarray(ref, np.float64) - shape.out_shift) / shape.out_scale
    return float(np.abs(y - y_ref).max() / np.abs(y_ref).max())


def e2e_selection(pred_gpu, pred_ref, arr, k):
    """End-to-end selection check: the GPU's chosen set (GPU select on GPU predictions, equal bit for
    bit to the oracle select on them) against the oracle select on the oracle's predictions.

    With e the largest |p_gpu - p_oracle| and t_k <= t_k+1 the oracle's k-th and (k+1)-th smallest
    keys, every job with oracle key below t_k - 2e must be chosen by the GPU and every job above
    t_k+1 + 2e must not be (a job that far from the cut cannot change sides by errors of at most e);
    this is asserted on every batch. When the gap t_k+1 - t_k exceeds 2e no job is in between, so
    the two sets must be equal. Returns the margin figures (the jobs inside the band are near-ties
    whose side the arithmetic does not fix)."""
    pred_gpu = np.asarray(pred_gpu, np.float32)
    pred_ref = np.asarray(pred_ref, np.float64)
    n = len(pred_ref)
    err = float(np.abs(pred_gpu.astype(np.float64) - pred_ref).max())
    got = set(oracle.oracle_select(pred_gpu, arr, k).tolist())
    exp = set(oracle.oracle_select(pred_ref, arr, k).tolist())
    if k >= n or k == 0:
        assert got == exp
        return dict(gap=float("inf"), max_err=err, margin_ok=True, sets_equal=True, near_ties=0)
    srt = np.sort(pred_ref)
    lo, hi = srt[k - 1] - 2 * err, srt[k] + 2 * err
    must = set(np.nonzero(pred_ref < lo)[0].tolist())
    never = set(np.nonzero(pred_ref > hi)[0].tolist())
    assert must <= got, sorted(must - got)
    assert not (never & got), sorted(never & got)
    gap = float(srt[k] - srt[k - 1])
    ok = gap > 2 * err
    if ok:
        assert got == exp, (gap, err)
    return dict(gap=gap, max_err=err, margin_ok=ok, sets_equal=got == exp, near_ties=n - len(must) - len(never))


def check_selection(pr, pred_gpu, d_arr, arr, k):
    """The GPU select on the GPU's predictions equals the oracle select on the same fp32 values."""
    idx, cnt = pr.select(torch.from_numpy(pred_gpu).cuda(), d_arr, k)
    torch.cuda.synchronize()
    m = int(cnt.item())
    got = idx.cpu().numpy()[:m]
    assert np.array_equal(got, oracle.oracle_select(pred_gpu, arr, k))


def test_embedding_layernorm_only():
    note("predict with zero layers (embedding + LayerNorm, pooling, head)")
    shape = dataclasses.replace(TINY, n_layers=0)
    W = make_weights(TINY, 1001)
    pr = Predictor(DeviceWeights(shape, {k: v for k, v in W.device.items()}))
    b = make_batch(W_TINY)
    pred, hid, _ = run(pr, b)
    m = dict(W.master)
    m["word"] = bf16_bits_to_f32(W.device["word"])   # the device tables are the bf16 roundings
    m["pos"] = bf16_bits_to_f32(W.device["pos"])
    ref_p, ref_h = oracle.oracle_forward(b.token_ids, b.cu_seqlens, m, shape)
    assert np.abs(hid - ref_h).max() < 1e-4
    assert rel_err(pred, ref_p).max() < 1e-5


def test_tiny_end_to_end():
    note("tiny predictor, all sequences, fp32 master weights in the oracle")
    W, pr = predictor(W_TINY.shape, W_TINY.weight_seed)
    b = make_batch(W_TINY)
    pred, hid, d_arr = run(pr, b)
    ref_p, ref_h = oracle.oracle_forward(b.token_ids, b.cu_seqlens, W.master, W_TINY.shape)
    herr = np.abs(hid - ref_h).max()
    perr = rel_err(pred, ref_p).max()
    yerr = y_rel(pred, ref_p, W_TINY.shape)
    note(f"tiny: hidden max-abs {herr:.3e}, pred max-rel {perr:.3e}, y rel {yerr:.3e}")
    assert herr <= HIDDEN_ATOL and perr <= PRED_RTOL and yerr <= Y_RTOL
    check_selection(pr, pred, d_arr, b.arrival_seq, W_TINY.batch_cap)
    sel = e2e_selection(pred, ref_p, b.arrival_seq, W_TINY.batch_cap)
    record(W_TINY.name, seqs=f"all {b.n}", hidden=herr, pred_rel=perr, y_rel=yerr, **sel)


@pytest.mark.parametrize("w,n", [(W_TINY_HEAD8, 8), (W_TINY_CLS_LIN8, 8), (W_TINY_HEAD8, 37)])
def test_tiny_deep_heads_end_to_end(w, n):
    """The paper's eight-layer heads (mean pooling + ReLU FC, Sec. 4.2; CLS + linear layers,
    Sec. 3.2) on every sequence; 37 sequences leave ragged groups in the head kernels."""
    w = dataclasses.replace(w, n_seqs=n, batch_cap=min(w.batch_cap, n))
    note(f"{w.name} with {n} sequences: eight-layer head, all sequences")
    W, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    pred, hid, d_arr = run(pr, b)
    ref_p, ref_h = oracle.oracle_forward(b.token_ids, b.cu_seqlens, W.master, w.shape)
    herr = np.abs(hid - ref_h).max()
    perr = rel_err(pred, ref_p).max()
    yerr = y_rel(pred, ref_p, w.shape)
    note(f"{w.name}: hidden max-abs {herr:.3e}, pred max-rel {perr:.3e}, y rel {yerr:.3e}, "
         f"pred spread {np.ptp(ref_p):.2f}")
    assert herr <= HIDDEN_ATOL and perr <= PRED_RTOL and yerr <= Y_RTOL
    check_selection(pr, pred, d_arr, b.arrival_seq, w.batch_cap)
    sel = e2e_selection(pred, ref_p, b.arrival_seq, w.batch_cap)
    record(f"{w.name} (n={n})", seqs=f"all {b.n}", hidden=herr, pred_rel=perr, y_rel=yerr, **sel)


def test_deterministic_and_packing_invariant():
    w = W_BERT_B64
    W, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    note("bert_base_b64 twice: bitwise equal")
    p1, h1, _ = run(pr, b)
    p2, h2, _ = run(pr, b)
    assert np.array_equal(p1, p2) and np.array_equal(h1, h2)
    note("bert_base_b64: sequences alone vs packed, bitwise equal")
    for s in (0, 17, 63):
        alone = pack([b.seq(s)])
        pa, ha, _ = run(pr, alone)
        assert pa[0] == p1[s]
        assert np.array_equal(ha, h1[b.cu_seqlens[s]:b.cu_seqlens[s + 1]])
    note("bert_base_b64: permuted batch gives permuted predictions")
    perm = np.random.default_rng(0).permutation(b.n)
    bp = pack([b.seq(int(i)) for i in perm])
    pp, _, _ = run(pr, bp, want_hidden=False)
    assert np.array_equal(pp, p1[perm])


def test_device_content_errors_are_flagged():
    W, pr = predictor(W_TINY.shape, W_TINY.weight_seed)
    b = make_batch(W_TINY)
    cases = []
    bad_ids = b.token_ids.copy()
    bad_ids[5] = W_TINY.shape.vocab + 3
    cases.append(("token id >= vocab", bad_ids, b.cu_seqlens, b.max_seqlen, E.ELIS_DEV_BAD_TOKEN))
    neg = b.token_ids.copy()
    neg[0] = -1
    cases.append(("negative token id", neg, b.cu_seqlens, b.max_seqlen, E.ELIS_DEV_BAD_TOKEN))
    cu = b.cu_seqlens.copy()
    cu[3], cu[4] = cu[4], cu[3]
    cases.append(("cu_seqlens not increasing", b.token_ids, cu, b.max_seqlen, E.ELIS_DEV_BAD_CU))
    cu0 = b.cu_seqlens.copy()
    cu0[0] = 2
    cases.append(("cu_seqlens[0] != 0", b.token_ids, cu0, b.max_seqlen, E.ELIS_DEV_BAD_CU))
    cases.append(("length above max_seqlen", b.token_ids, b.cu_seqlens, int(b.lengths.min()), E.ELIS_DEV_LONG_SEQ))
    for what, ids, cu_, msl, bit in cases:
        note(f"content error: {what}")
        pred, _ = pr.predict(dev(ids), dev(cu_), msl)
        st, bits = pr.status()
        assert st == E.ELIS_EDEVICE and bits & bit, (what, st, bits)
    note("valid batch after errors: status clears")
    run(pr, b)


@pytest.mark.parametrize("w", [W_TINY, W_TINY_HEAD8], ids=lambda w: w.name)
def test_timing_counts_class_launches_and_keeps_results(w):
    """The opt-in per-class timing: one count per class launch (the head of mean pooling enqueues
    several kernels and still counts once), positive times, and bitwise the same predictions and
    selection as an untimed pass."""
    note(f"timing hook {w.name}")
    _, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    ids, cu, arr = upload_batch(b)
    p0, _ = pr.predict(ids, cu, b.max_seqlen)
    i0, c0 = pr.select(p0, arr, w.batch_cap)
    torch.cuda.synchronize()
    E.elis_timing_reset()
    E.elis_timing_enable((1 << len(E.KERNEL_CLASSES)) - 1)
    try:
        for _ in range(2):
            p1, _ = pr.predict(ids, cu, b.max_seqlen)
            i1, c1 = pr.select(p1, arr, w.batch_cap)
        torch.cuda.synchronize()
    finally:
        E.elis_timing_enable(0)
    L = w.shape.n_layers
    want = {"seqmap": 1, "embed_ln": 1, "gemm_qkv": L, "attention": L, "gemm_o": L, "layernorm": 2 * L,
            "gemm_ffn1": L, "gemm_ffn2": L, "pool_head": 1, "select": 1}
    for name in E.KERNEL_CLASSES:
        st, nl, ms = E.elis_timing_read(E.K[name])
        assert st == E.ELIS_OK
        assert nl == 2 * want.get(name, 0), name
        assert (ms > 0) == (nl > 0), name
    E.elis_timing_reset()
    assert E.elis_timing_read(E.K["gemm_qkv"])[1] == 0
    assert torch.equal(p0, p1)
    assert int(c0.item()) == int(c1.item())
    assert torch.equal(i0[:int(c0.item())], i1[:int(c1.item())])


def test_timing_stride_samples_class_launches():
    """With a stride s the timing covers launch 0, s, 2s, ... of each class since the last reset,
    counted across forward passes (so a stride coprime to the layer count rotates over the layers)."""
    w = W_TINY
    note(f"timing stride {w.name}")
    _, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    ids, cu, arr = upload_batch(b)
    L, passes, stride = w.shape.n_layers, 5, 3
    E.elis_timing_reset()
    assert E.elis_timing_stride(stride) == E.ELIS_OK
    E.elis_timing_enable((1 << E.K["gemm_ffn2"]) | (1 << E.K["layernorm"]))
    try:
        for _ in range(passes):
            pr.predict(ids, cu, b.max_seqlen)
        torch.cuda.synchronize()
    finally:
        E.elis_timing_enable(0)
        E.elis_timing_stride(1)
    for name, per_pass in (("gemm_ffn2", L), ("layernorm", 2 * L)):
        st, nl, ms = E.elis_timing_read(E.K[name])
        assert st == E.ELIS_OK
        assert nl == -(-passes * per_pass // stride), name
        assert ms > 0
    assert E.elis_timing_read(E.K["gemm_qkv"])[1] == 0
    E.elis_timing_reset()


@pytest.mark.parametrize("w", [W_TINY, W_TINY_CLS_LIN8, W_BERT_B64, W_TINY_HEAD8], ids=lambda w: w.name)
def test_cls_tail_is_bit_identical(w):
    """Without a hidden-state output and with CLS pooling, the last layer runs on the CLS rows
    only (after its full QKV product); the predictions must equal the full pass bit for bit.
    Mean pooling (tiny_head8) always runs the full pass: both calls agree there too."""
    note(f"CLS-only last layer vs full pass: {w.name}")
    _, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    p_full, h_full, _ = run(pr, b, want_hidden=True)
    p_tail, h_tail, _ = run(pr, b, want_hidden=False)
    assert h_tail is None and h_full is not None
    assert np.array_equal(p_full.view(np.uint32), p_tail.view(np.uint32))
    if w.shape.pooling == 0:
        # and a batch of length-1 sequences (n = T: the one-row-per-sequence buffers are full-size)
        ones = pack([b.seq(s)[:1] for s in range(b.n)])
        p1, _, _ = run(pr, ones, want_hidden=True)
        p2, _, _ = run(pr, ones, want_hidden=False)
        assert np.array_equal(p1.view(np.uint32), p2.view(np.uint32))


def test_hip_graph_replay_matches_eager():
    """elis_predict_remaining + elis_isrtf_select only enqueue kernels (no allocation, memset or
    synchronisation), so a round can be captured into a HIP graph. Every replay, with eager
    library work and synchronisations between replays, must give the eager results bit for bit."""
    w = W_BERT_B64
    note("HIP graph capture of predict + select (bert_base_b64)")
    _, pr = predictor(w.shape, w.weight_seed)
    b = make_batch(w)
    ids, cu, arr = upload_batch(b)
    other = make_batch(dataclasses.replace(w, data_seed=w.data_seed + 5))
    o_ids, o_cu, _ = upload_batch(other)
    pred = torch.empty(b.n, dtype=torch.float32, device="cuda")
    idx = torch.full((w.batch_cap,), -1, dtype=torch.int32, device="cuda")
    cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
    # eager reference; the same call also sizes the cached workspaces before capture
    pr.predict(ids, cu, b.max_seqlen, out_pred=pred)
    pr.select(pred, arr, w.batch_cap, idx, cnt)
    torch.cuda.synchronize()
    ref_pred, ref_idx, ref_cnt = pred.clone(), idx.clone(), cnt.clone()
    pr.predict(o_ids, o_cu, other.max_seqlen)  # a larger workspace now, before capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            pr.predict(ids, cu, b.max_seqlen, out_pred=pred)
            pr.select(pred, arr, w.batch_cap, idx, cnt)
    torch.cuda.current_stream().wait_stream(side)
    for rep in range(4):
        pred.fill_(float("nan"))
        idx.fill_(-7)
        cnt.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(pred.view(torch.int32), ref_pred.view(torch.int32)), rep
        assert torch.equal(cnt, ref_cnt) and torch.equal(idx, ref_idx), rep
        # eager work on another batch between replays (it shares the predictor's workspace)
        p_other, _ = pr.predict(o_ids, o_cu, other.max_seqlen)
        torch.cuda.synchronize()
        assert torch.isfinite(p_other).all()
    st, bits = pr.status()
    assert st == E.ELIS_OK, (st, bits)
