"""Per-kernel parity of libelis against the fp64 oracle, through the C ABI.

Tolerances follow from the arithmetic: operands are bf16 (8-bit significand),
accumulation is fp32, and bf16 outputs carry one final rounding of relative
size <= 2^-8 (half a unit in the last of 8 significant bits).
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2505_09142_amd import _elis as E
from tests.gpu_util import bf16_to_f64, dev, host_u16, note, ok, stream, workspace
from workloads import BERT_BASE, BERT_BASE_HEAD8, TINY, TINY_CLS_LIN8, TINY_HEAD8, f32_to_bf16_bits, pack

pytestmark = pytest.mark.gpu

U32 = lambda *v: np.array(v, dtype=np.uint32).view(np.float32)
SPECIAL_BITS = U32(0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 0xFFC00000, 0x7F800001,
                   0xFF812345, 0x00000001, 0x80000001, 0x007FFFFF, 0x807FFFFF, 0x3F800000, 0x3F800000,
                   0xBF800000, 0x7F7FFFFF, 0xFF7FFFFF)


def _preds(kind: str, n: int, rng) -> np.ndarray:
    if kind == "normal":
        return (rng.standard_normal(n) * 100 + 250).astype(np.float32)
    if kind == "ties":
        return rng.integers(0, 4, size=n).astype(np.float32)
    if kind == "special":
        return rng.choice(SPECIAL_BITS, size=n)
    if kind == "equal":
        return np.full(n, 7.5, np.float32)
    raise ValueError(kind)


SELECT_CASES = [(n, kind) for n in (1, 2, 8, 64, 255, 256, 1000, 1024) for kind in ("normal", "ties", "special")]
SELECT_CASES += [(n, kind) for n in (1025, 3000, 4096, 8192) for kind in ("normal", "ties", "special", "equal")]
SELECT_CASES += [(64, "equal"), (1024, "equal")]


@pytest.mark.parametrize("n,kind", SELECT_CASES)
def test_select_bit_exact(n, kind):
    rng = np.random.default_rng(n * 7 + len(kind))
    pred = _preds(kind, n, rng)
    arr = rng.integers(0, max(2, n // 2), size=n).astype(np.int64)   # repeated arrival values too
    d_pred, d_arr = dev(pred), dev(arr)
    buf, ws, wsb = workspace(E.elis_select_workspace_bytes(n))
    for k in sorted({0, 1, n // 2, n, n + 5}):
        note(f"select n={n} kind={kind} k={k}")
        idx = torch.full((max(1, k),), -1, dtype=torch.int32, device="cuda")
        cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        ok(E.elis_isrtf_select(d_pred.data_ptr(), d_arr.data_ptr(), n, k, idx.data_ptr(), cnt.data_ptr(), ws, wsb,
                               stream()), "select")
        torch.cuda.synchronize()
        m = min(k, n)
        assert int(cnt.item()) == m
        got = idx.cpu().numpy()[:m]
        exp = oracle.oracle_select(pred, arr, k)
        assert np.array_equal(got, exp), f"n={n} kind={kind} k={k}"
        st, bits = E.elis_read_status(ws, stream())
        assert st == E.ELIS_OK and bits == 0


def test_select_worked_example():
    import json, os
    cases = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "srtf_two_requests.json")))["cases"]
    buf, ws, wsb = workspace(256)
    for c in cases:
        note(f"select golden: {c['what']}")
        pred = dev(np.array(c["pred"], np.float32))
        arr = dev(np.array(c["arrival_seq"], np.int64))
        idx = torch.full((2,), -1, dtype=torch.int32, device="cuda")
        cnt = torch.zeros(1, dtype=torch.int32, device="cuda")
        ok(E.elis_isrtf_select(pred.data_ptr(), arr.data_ptr(), 2, c["batch_cap"], idx.data_ptr(), cnt.data_ptr(),
                               ws, wsb, stream()))
        torch.cuda.synchronize()
        assert idx.cpu().numpy()[:int(cnt.item())].tolist() == c["selected"]


# ------------------------------------------------------------------------------ select, large n
# Above 8192 jobs the device-wide radix selection runs; "ties" (four distinct values) and
# "equal" give tie sets above 8192, which exercises the selection among ties by arrival.
SELECT_LARGE_CASES = [(8193, "normal"), (8193, "equal"), (20000, "special"), (100003, "ties"),
                      (100003, "normal"), (1 << 20, "normal"), (1 << 20, "special")]


def _run_select(d_pred, d_arr, n, k, ws, wsb):
    idx = torch.full((max(1, k),), -1, dtype=torch.int32, device="cuda")
    cnt = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ok(E.elis_isrtf_select(d_pred.data_ptr(), d_arr.data_ptr(), n, k, idx.data_ptr(), cnt.data_ptr(), ws, wsb,
                           stream()), "select")
    torch.cuda.synchronize()
    assert int(cnt.item()) == min(k, n)
    st, bits = E.elis_read_status(ws, stream())
    assert st == E.ELIS_OK and bits == 0
    return idx.cpu().numpy()[:min(k, n)]


@pytest.mark.parametrize("n,kind", SELECT_LARGE_CASES)
def test_select_large_bit_exact(n, kind):
    rng = np.random.default_rng(n + 31 * len(kind))
    pred = _preds(kind, n, rng)
    arr = rng.integers(0, max(2, n // 2), size=n).astype(np.int64)
    order = np.asarray(oracle.oracle_order(pred, arr), dtype=np.int32)
    d_pred, d_arr = dev(pred), dev(arr)
    buf, ws, wsb = workspace(E.elis_select_workspace_bytes(n))
    for k in (0, 1, 37, 8192):
        note(f"select large n={n} kind={kind} k={k}")
        got = _run_select(d_pred, d_arr, n, k, ws, wsb)
        assert np.array_equal(got, order[:min(k, n)]), f"n={n} kind={kind} k={k}"


def _order_key_np(pred):
    u = pred.view(np.uint32).copy()
    u[u == 0x80000000] = 0
    key = np.where(u & 0x80000000, ~u, u | 0x80000000).astype(np.uint32)
    key[np.isnan(pred)] = 0xFFFFFFFF
    return key


@pytest.mark.parametrize("n,kind,k", [(1 << 24, "normal", 64), (1 << 24, "normal", 8192), (1 << 22, "ties", 500)])
def test_select_large_properties(n, kind, k):
    """At sizes the sort-based oracle does not reach: the output is strictly increasing in
    the total order (key, arrival, index), and exactly k-1 jobs precede its last element."""
    rng = np.random.default_rng(n + k)
    pred = _preds(kind, n, rng)
    arr = rng.integers(0, n, size=n).astype(np.int64)
    note(f"select properties n={n} kind={kind} k={k}")
    buf, ws, wsb = workspace(E.elis_select_workspace_bytes(n))
    got = _run_select(dev(pred), dev(arr), n, k, ws, wsb)
    key = _order_key_np(pred)
    gk, ga = key[got].astype(np.int64), arr[got]
    inc = (gk[1:] > gk[:-1]) | ((gk[1:] == gk[:-1]) & ((ga[1:] > ga[:-1]) | ((ga[1:] == ga[:-1]) & (got[1:] > got[:-1]))))
    assert inc.all()
    lk, la, li = int(gk[-1]), int(ga[-1]), int(got[-1])
    idx = np.arange(n)
    before = (key < lk) | ((key == lk) & ((arr < la) | ((arr == la) & (idx < li))))
    assert int(before.sum()) == k - 1


# ------------------------------------------------------------------------------ LayerNorm

@pytest.mark.parametrize("rows,d", [(1, 64), (7, 128), (1000, 768), (333, 1024), (65, 2048)])
def test_layernorm(rows, d):
    note(f"layernorm rows={rows} d={d}")
    rng = np.random.default_rng(rows + d)
    x = (rng.standard_normal((rows, d)) * 3 + 1.5).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    b = (0.1 * rng.standard_normal(d)).astype(np.float32)
    eps = 1e-5
    o32 = torch.empty((rows, d), dtype=torch.float32, device="cuda")
    o16 = torch.empty((rows, d), dtype=torch.int16, device="cuda")
    d_x, d_g, d_b = dev(x), dev(g), dev(b)  # keep the uploads alive until the kernel has run
    ok(E.elis_layernorm(d_x.data_ptr(), d_g.data_ptr(), d_b.data_ptr(), rows, d, eps, o32.data_ptr(),
                        o16.data_ptr(), stream()))
    torch.cuda.synchronize()
    ref = oracle.layer_norm(x.astype(np.float64), g, b, eps)
    err32 = np.abs(o32.cpu().numpy() - ref)
    assert err32.max() < 2e-5 * (1 + np.abs(ref).max()), err32.max()
    got16 = bf16_to_f64(host_u16(o16))
    assert np.all(np.abs(got16 - ref) <= 2.0 ** -8 * np.abs(ref) + 2e-5)


# ------------------------------------------------------------------------------ GEMM

GEMM_CASES = [(1, 64, 64), (37, 128, 64), (300, 384, 128), (1000, 768, 768), (129, 3072, 768),
              (517, 768, 3072), (2048, 2304, 768), (77, 192, 256), (64, 256, 64), (300, 512, 128), (1111, 1024, 4096)]


@pytest.mark.parametrize("epi", [E.ELIS_EPI_BIAS_BF16, E.ELIS_EPI_BIAS_GELU_BF16, E.ELIS_EPI_BIAS_RES_F32])
@pytest.mark.parametrize("m,n,k", GEMM_CASES)
def test_linear(m, n, k, epi):
    note(f"linear m={m} n={n} k={k} epi={epi}")
    rng = np.random.default_rng(m * 31 + n + k + epi)
    xb = f32_to_bf16_bits(rng.standard_normal((m, k)).astype(np.float32))
    wb = f32_to_bf16_bits((rng.standard_normal((n, k)) * 0.05).astype(np.float32))
    bias = (rng.standard_normal(n) * 0.1).astype(np.float32)
    res = rng.standard_normal((m, n)).astype(np.float32)
    x64, w64 = bf16_to_f64(xb), bf16_to_f64(wb)
    pre = x64 @ w64.T + bias
    mag = np.abs(x64) @ np.abs(w64).T                    # bound on fp32 accumulation error scale
    if epi == E.ELIS_EPI_BIAS_RES_F32:
        out = torch.empty((m, n), dtype=torch.float32, device="cuda")
        d_res = dev(res)
        rp = d_res.data_ptr()
    else:
        out = torch.empty((m, n), dtype=torch.int16, device="cuda")
        rp = None
    d_x, d_w, d_bias = dev(xb), dev(wb), dev(bias)  # keep the uploads alive until the kernel has run
    ok(E.elis_linear(d_x.data_ptr(), d_w.data_ptr(), d_bias.data_ptr(), rp, m, n, k, epi,
                     out.data_ptr(), stream()))
    torch.cuda.synchronize()
    acc_tol = 1e-5 * mag + 1e-6
    if epi == E.ELIS_EPI_BIAS_RES_F32:
        ref = pre + res
        got = out.cpu().numpy().astype(np.float64)
        assert np.all(np.abs(got - ref) <= acc_tol + 1e-6 * np.abs(ref))
    else:
        ref = oracle.gelu(pre) if epi == E.ELIS_EPI_BIAS_GELU_BF16 else pre
        got = bf16_to_f64(host_u16(out))
        assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1.2 * acc_tol), np.abs(got - ref).max()


def test_gelu_epilogue_sweep():
    """The GELU epilogue over a dense sweep of pre-activations, tails and clamp included: with
    x = 0 and W = 0 the product is exactly the bias, so each output is bf16(GELU(bias[n]))."""
    m, n, k = 3, 8192, 64
    special = np.array([0.0, -0.0, 5.0, -5.0, 4.9999, -4.9999, 5.0001, -5.0001, 20.0, -20.0, 100.0, -100.0,
                        1e4, -1e4, 1e-30, -1e-30, 1e-3, -1e-3, 0.5, -0.5], np.float32)
    sweep = np.linspace(-8.0, 8.0, n - special.size, dtype=np.float32)
    bias = np.concatenate([sweep, special]).astype(np.float32)
    note(f"gelu epilogue sweep m={m} n={n} k={k}")
    d_x = dev(np.zeros((m, k), np.uint16))
    d_w = dev(np.zeros((n, k), np.uint16))
    d_bias = dev(bias)
    out = torch.empty((m, n), dtype=torch.int16, device="cuda")
    ok(E.elis_linear(d_x.data_ptr(), d_w.data_ptr(), d_bias.data_ptr(), None, m, n, k, E.ELIS_EPI_BIAS_GELU_BF16,
                     out.data_ptr(), stream()))
    torch.cuda.synchronize()
    got = bf16_to_f64(host_u16(out))
    ref = oracle.gelu(bias.astype(np.float64))
    err = np.abs(got - ref[None, :])
    assert np.all(err <= 2.0 ** -8 * np.abs(ref)[None, :] + 2e-6), (err.max(), bias[np.argmax(err.max(axis=0))])
    assert np.array_equal(got[0], got[1]) and np.array_equal(got[0], got[2])


# ------------------------------------------------------------------------------ attention

ATT_LENS = [
    [1],
    [5, 1, 17],
    [63, 64, 65],
    [127, 128, 129, 1, 300],
    [512, 200, 511],
    [1000, 33],
]


def attention_bound(q, k, v, heads, ref):
    """Per-element error bound of the GPU attention output, from its arithmetic.

    The kernel rounds each softmax weight p_ij to bf16 (relative error d_ij, |d_ij| <= 2^-8) and
    normalises by the sum of the same rounded weights, so the weights it applies are
    w_ij (1 + d_ij) / (1 + sum_j w_ij d_ij); their deviation from the exact weights w_ij is at most
    w_ij |d_ij - mean d| / (1 - 2^-8) <= 2^-7 w_ij (1 + 2^-7). The output o_ic = sum_j w_ij v_jc
    is therefore off by at most 2^-7 (1 + 2^-7) sum_j w_ij |v_jc|, plus the final bf16 rounding
    (2^-8 of the value), plus fp32 scores, exponentials and accumulation (taken as 2^-12 of
    sum_j w_ij |v_jc|, a generous allowance: fp32 score errors of sharp rows change a weight by
    ~2^-14 of itself). The bound is per query row and per column: it scales with the row's own
    attention-weighted |v|, not with the largest value of the sequence.
    """
    n, D = q.shape
    dh = D // heads
    A = np.empty((n, D))
    for h in range(heads):
        c = slice(h * dh, (h + 1) * dh)
        w = oracle.softmax_rows((q[:, c] @ k[:, c].T) / np.sqrt(dh))
        A[:, c] = w @ np.abs(v[:, c])
    s = 2.0 ** -7 * (1 + 2.0 ** -7) + 2.0 ** -12
    return s * A + 2.0 ** -8 * (np.abs(ref) + s * A) + 1e-30


def _attention_case(lens, heads, dh, sharp, seed):
    rng = np.random.default_rng(seed)
    T = int(sum(lens))
    D = heads * dh
    qkv = rng.standard_normal((T, 3 * D)).astype(np.float32)
    if sharp:
        qkv[:, :D] *= 6.0  # peaked softmax: large score gaps
    qkv_b = f32_to_bf16_bits(qkv)
    b = pack([np.zeros(L, np.int32) for L in lens])
    return qkv_b, b, T, D


@pytest.mark.parametrize("dh,heads", [(64, 2), (32, 4), (64, 12)])
@pytest.mark.parametrize("lens", ATT_LENS)
@pytest.mark.parametrize("sharp", [False, True])
def test_attention(lens, dh, heads, sharp):
    note(f"attention lens={lens} dh={dh} heads={heads} sharp={sharp}")
    qkv_b, b, T, D = _attention_case(lens, heads, dh, sharp, seed=sum(lens) + dh + heads + sharp)
    n = len(lens)
    out = torch.empty((T, D), dtype=torch.int16, device="cuda")
    buf, ws, wsb = workspace(E.elis_attention_workspace_bytes(n, T))
    d_cu, d_qkv = dev(b.cu_seqlens), dev(qkv_b)
    ok(E.elis_attention(d_qkv.data_ptr(), d_cu.data_ptr(), n, T, max(lens), heads, dh, out.data_ptr(), ws,
                        wsb, stream()))
    st, bits = E.elis_read_status(ws, stream())
    assert st == E.ELIS_OK and bits == 0
    got = bf16_to_f64(host_u16(out))
    q64 = bf16_to_f64(qkv_b)
    worst = 0.0
    for s in range(n):
        a, e = b.cu_seqlens[s], b.cu_seqlens[s + 1]
        q, k, v = q64[a:e, :D], q64[a:e, D:2 * D], q64[a:e, 2 * D:]
        ref = oracle.self_attention(q, k, v, heads)
        bound = attention_bound(q, k, v, heads, ref)
        err = np.abs(got[a:e] - ref)
        worst = max(worst, float((err / bound).max()))
        assert np.all(err <= bound), (s, float((err / bound).max()))
    note(f"attention: largest error / per-element bound {worst:.3f}")


def test_attention_single_token_is_value():
    note("attention single-token sequences")
    heads, dh = 2, 64
    lens = [1] * 9
    qkv_b, b, T, D = _attention_case(lens, heads, dh, False, 3)
    out = torch.empty((T, D), dtype=torch.int16, device="cuda")
    buf, ws, wsb = workspace(E.elis_attention_workspace_bytes(9, T))
    d_qkv, d_cu = dev(qkv_b), dev(b.cu_seqlens)
    ok(E.elis_attention(d_qkv.data_ptr(), d_cu.data_ptr(), 9, T, 1, heads, dh, out.data_ptr(), ws,
                        wsb, stream()))
    torch.cuda.synchronize()
    # softmax over one key is exactly 1, so the output is the value row, bit for bit
    assert np.array_equal(host_u16(out), qkv_b[:, 2 * D:])


@pytest.mark.parametrize("lens", [[1000, 33], [512, 200, 511], [127, 128, 129, 1, 300]])
@pytest.mark.parametrize("sharp", [False, True])
def test_attention_normalisation_is_exact(lens, sharp):
    """Value columns that are one constant c (a power of two) for every key of a sequence: the
    kernel's output there is (sum_j p_ij c) / (sum_j p_ij) over the same bf16 weights, both sums
    accumulated by the same matrix-core instruction and rescaled by the same factors, so it must
    be c exactly, on every row, whatever the scores (a wrong row sum, a missed rescale of the
    accumulators or of the sum after the running maximum moves would show here)."""
    heads, dh = 2, 64
    note(f"attention normalisation lens={lens} sharp={sharp}")
    qkv_b, b, T, D = _attention_case(lens, heads, dh, sharp, seed=sum(lens) + 17 * sharp)
    consts = {2 * D + 3: 1.0, 2 * D + 40: -2.0, 2 * D + dh + 5: 0.5, 2 * D + dh + 63: 4.0}
    qkv_b = qkv_b.copy()
    for col, c in consts.items():
        qkv_b[:, col] = f32_to_bf16_bits(np.full(T, c, np.float32))
    n = len(lens)
    out = torch.empty((T, D), dtype=torch.int16, device="cuda")
    buf, ws, wsb = workspace(E.elis_attention_workspace_bytes(n, T))
    d_cu, d_qkv = dev(b.cu_seqlens), dev(qkv_b)
    ok(E.elis_attention(d_qkv.data_ptr(), d_cu.data_ptr(), n, T, max(lens), heads, dh, out.data_ptr(), ws,
                        wsb, stream()))
    torch.cuda.synchronize()
    got = bf16_to_f64(host_u16(out))
    for col, c in consts.items():
        assert np.all(got[:, col - 2 * D] == c), (col, c)


def test_attention_flags_bad_cu_without_faulting():
    note("attention with malformed cu_seqlens (clamped, flagged)")
    heads, dh = 2, 32
    qkv_b = f32_to_bf16_bits(np.ones((20, 3 * heads * dh), np.float32))
    cu = np.array([0, 10, 5, 20], np.int32)  # not increasing
    out = torch.zeros((20, heads * dh), dtype=torch.int16, device="cuda")
    buf, ws, wsb = workspace(E.elis_attention_workspace_bytes(3, 20))
    d_qkv, d_cu = dev(qkv_b), dev(cu)
    ok(E.elis_attention(d_qkv.data_ptr(), d_cu.data_ptr(), 3, 20, 16, heads, dh, out.data_ptr(), ws, wsb,
                        stream()))
    st, bits = E.elis_read_status(ws, stream())
    assert st == E.ELIS_EDEVICE and bits & E.ELIS_DEV_BAD_CU


@pytest.mark.parametrize("epi", [E.ELIS_EPI_BIAS_RES_F32, E.ELIS_EPI_BIAS_GELU_BF16, E.ELIS_EPI_BIAS_BF16])
def test_linear_large_m_sampled(epi):
    """Token counts of the 100-round workload (~50K-110K rows) take other tile configurations;
    checked on sampled rows (first, last, ragged tail and random ones)."""
    m, n, k = 50001, 768 if epi == E.ELIS_EPI_BIAS_RES_F32 else 1024, 3072 if epi == E.ELIS_EPI_BIAS_RES_F32 else 768
    note(f"linear large m={m} n={n} k={k} epi={epi}")
    rng = np.random.default_rng(epi + 7)
    xb = f32_to_bf16_bits(rng.standard_normal((m, k), dtype=np.float32))
    wb = f32_to_bf16_bits((rng.standard_normal((n, k), dtype=np.float32) * 0.05))
    bias = (rng.standard_normal(n) * 0.1).astype(np.float32)
    res = rng.standard_normal((m, n), dtype=np.float32)
    d_x, d_w, d_bias, d_res = dev(xb), dev(wb), dev(bias), dev(res)
    f32 = epi == E.ELIS_EPI_BIAS_RES_F32
    out = torch.empty((m, n), dtype=torch.float32 if f32 else torch.int16, device="cuda")
    ok(E.elis_linear(d_x.data_ptr(), d_w.data_ptr(), d_bias.data_ptr(), d_res.data_ptr() if f32 else None, m, n, k,
                     epi, out.data_ptr(), stream()))
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, m - 1, m - 2, m - 17], rng.integers(0, m, 300)]))
    x64, w64 = bf16_to_f64(xb[rows]), bf16_to_f64(wb)
    pre = x64 @ w64.T + bias
    acc_tol = 1e-5 * (np.abs(x64) @ np.abs(w64).T) + 1e-6
    if f32:
        got = out[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
        ref = pre + res[rows]
        assert np.all(np.abs(got - ref) <= acc_tol + 1e-6 * np.abs(ref))
    else:
        got = bf16_to_f64(host_u16(out[torch.from_numpy(rows).cuda()]))
        ref = oracle.gelu(pre) if epi == E.ELIS_EPI_BIAS_GELU_BF16 else pre
        assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1.2 * acc_tol)


def test_linear_split_plans_agree_bitwise():
    """Products whose launch plans differ (one launch of 64 x 128, 128 x 128 or 256 x 256 tiles, or
    large tiles over whole rounds plus a second launch of small tiles over the remaining rows) give
    the same bits on the rows they share."""
    rng = np.random.default_rng(78)
    for n, k, epi, ms in ((768, 3072, E.ELIS_EPI_BIAS_RES_F32, (300, 5000, 23931, 30000)),
                          (2304, 768, E.ELIS_EPI_BIAS_BF16, (700, 6000, 23931, 26000)),
                          (3072, 768, E.ELIS_EPI_BIAS_GELU_BF16, (3000, 12000, 23931))):
        plans = {m: E.elis_linear_plan(m, n, k, epi)[1] for m in ms}
        assert len(set(plans.values())) >= 3, plans
        assert any(p[3] < m for m, p in plans.items()), plans   # at least one split plan
        m_max = max(ms)
        note(f"linear split plans n={n} k={k} epi={epi} plans={plans}")
        xb = f32_to_bf16_bits(rng.standard_normal((m_max, k), dtype=np.float32))
        wb = f32_to_bf16_bits(rng.standard_normal((n, k), dtype=np.float32) * 0.05)
        bias = (rng.standard_normal(n) * 0.1).astype(np.float32)
        f32 = epi == E.ELIS_EPI_BIAS_RES_F32
        res = rng.standard_normal((m_max, n), dtype=np.float32) if f32 else None
        d_x, d_w, d_bias = dev(xb), dev(wb), dev(bias)
        d_res = dev(res) if f32 else None
        outs = {}
        for m in ms:
            out = torch.empty((m, n), dtype=torch.float32 if f32 else torch.int16, device="cuda")
            ok(E.elis_linear(d_x.data_ptr(), d_w.data_ptr(), d_bias.data_ptr(), d_res.data_ptr() if f32 else None,
                             m, n, k, epi, out.data_ptr(), stream()))
            torch.cuda.synchronize()
            outs[m] = out.cpu().numpy().view(np.uint32 if f32 else np.uint16)
        ref = outs[m_max]
        for m in ms:
            assert np.array_equal(outs[m], ref[:m]), (m, plans[m])
        # every tile configuration and split forced through elis_linear_with_plan: the same bits
        m = m_max
        forced = [(128, 128, 2, m, 0, 0, 0), (64, 128, 2, m, 0, 0, 0), (64, 128, 1, m, 0, 0, 0),
                  (64, 64, 4, m, 0, 0, 0), (64, 64, 2, m, 0, 0, 0),
                  (128, 128, 2, 8192, 64, 128, 1), (64, 128, 2, 4096, 128, 128, 2), (128, 128, 2, 8192, 64, 64, 4)]
        if n % 256 == 0:
            forced += [(256, 256, 1, m, 0, 0, 0), (256, 256, 1, 4096, 64, 128, 2), (256, 256, 1, 8192, 128, 128, 2)]
        for plan in forced:
            note(f"  forced plan {plan}")
            out = torch.empty((m, n), dtype=torch.float32 if f32 else torch.int16, device="cuda")
            ok(E.elis_linear_with_plan(d_x.data_ptr(), d_w.data_ptr(), d_bias.data_ptr(),
                                       d_res.data_ptr() if f32 else None, m, n, k, epi, plan, out.data_ptr(), stream()))
            torch.cuda.synchronize()
            assert np.array_equal(out.cpu().numpy().view(np.uint32 if f32 else np.uint16), ref), plan
        # and the largest against the fp64 product on sampled rows
        rows = np.unique(np.concatenate([[0, m_max - 1], rng.integers(0, m_max, 200)]))
        x64, w64 = bf16_to_f64(xb[rows]), bf16_to_f64(wb)
        pre = x64 @ w64.T + bias
        acc_tol = 1e-5 * (np.abs(x64) @ np.abs(w64).T) + 1e-6
        if f32:
            got = ref[rows].view(np.float32).astype(np.float64)
            assert np.all(np.abs(got - (pre + res[rows])) <= acc_tol + 1e-6 * np.abs(pre + res[rows]))
        else:
            got = bf16_to_f64(ref[rows].view(np.uint16))
            exp = oracle.gelu(pre) if epi == E.ELIS_EPI_BIAS_GELU_BF16 else pre
            assert np.all(np.abs(got - exp) <= 2.0 ** -8 * np.abs(exp) + 1.2 * acc_tol)


def test_linear_routes_agree_bitwise():
    """Shapes routed to different tile configurations accumulate every output element in the same
    order with the same instruction and the same epilogue arithmetic: a row (column) computed by
    one configuration equals the same row (column) computed by another, bit for bit. This is what
    keeps the predictor's outputs independent of how many tokens are packed with a sequence."""
    rng = np.random.default_rng(77)
    cases = [  # (m_a, n_a, m_b, n_b, k, epi): a's output is the top-left corner of b's
        (23931, 768, 36864, 768, 3072, E.ELIS_EPI_BIAS_RES_F32),   # 128x128 pairs vs 256x256
        (23931, 768, 40960, 768, 768, E.ELIS_EPI_BIAS_RES_F32),
        (3000, 384, 3000, 512, 768, E.ELIS_EPI_BIAS_GELU_BF16),     # direct-to-LDS 128x128 vs 256x256
        (3000, 384, 3000, 512, 768, E.ELIS_EPI_BIAS_BF16),
    ]
    for m_a, n_a, m_b, n_b, k, epi in cases:
        note(f"linear routes m={m_a}/{m_b} n={n_a}/{n_b} k={k} epi={epi}")
        xb = f32_to_bf16_bits(rng.standard_normal((m_b, k), dtype=np.float32))
        wb = f32_to_bf16_bits(rng.standard_normal((n_b, k), dtype=np.float32) * 0.05)
        bias = (rng.standard_normal(n_b) * 0.1).astype(np.float32)
        f32 = epi == E.ELIS_EPI_BIAS_RES_F32
        res = rng.standard_normal((m_b, n_b), dtype=np.float32) if f32 else None
        outs = []
        for m, n in ((m_a, n_a), (m_b, n_b)):
            d_x, d_w, d_bias = dev(xb[:m]), dev(wb[:n]), dev(bias[:n])
            d_res = dev(np.ascontiguousarray(res[:m, :n])) if f32 else None
            out = torch.empty((m, n), dtype=torch.float32 if f32 else torch.int16, device="cuda")
            ok(E.elis_linear(d_x.data_ptr(), d_w.data_ptr(), d_bias.data_ptr(), d_res.data_ptr() if f32 else None,
                             m, n, k, epi, out.data_ptr(), stream()))
            torch.cuda.synchronize()
            outs.append(out.cpu().numpy())
        a, b = outs
        assert np.array_equal(a.view(np.uint32 if f32 else np.uint16),
                              np.ascontiguousarray(b[:m_a, :n_a]).view(np.uint32 if f32 else np.uint16))


# ----------------------------------------------------------------------------- pooling + head

HEAD_CASES = [
    # (shape, sequence lengths): CLS / mean pooling; linear, 2-layer and 8-layer heads; ragged counts
    (TINY, [16, 1, 64, 37, 5, 128, 2, 9]),
    (BERT_BASE, [1, 200, 512, 63, 64, 65]),
    (TINY_HEAD8, [16, 1, 64, 37, 5, 128, 2, 9, 65, 127, 3]),
    (TINY_CLS_LIN8, [4] * 37),
    (BERT_BASE_HEAD8, [1, 64, 65, 129, 512, 300, 17] * 10),
    (dataclasses.replace(BERT_BASE, name="bert_base_mean_linear", pooling=1, head_hidden=0), [1, 64, 65, 511, 7]),
    # widths off the matrix-core tile: 20 (no layer is a multiple of 16 units: every hidden layer on
    # the one-wave-per-unit kernel) and 48 (the first layer on the tile, the 48-input middle layers not)
    (dataclasses.replace(TINY_HEAD8, name="tiny_head8_w20", head_hidden=20), [16, 1, 64, 37, 5]),
    (dataclasses.replace(TINY_HEAD8, name="tiny_head8_w48", head_hidden=48), [16, 1, 64, 37, 5, 19, 33]),
]


@pytest.mark.parametrize("shape,lens", HEAD_CASES, ids=lambda v: v.name if hasattr(v, "name") else f"n{len(v)}")
def test_pool_head(shape, lens):
    """elis_pool_head on random final hidden states against the oracle's pooling and head, for every
    sequence. fp32 throughout: the bound is 1e-4 of the largest |y| (fp32 dot products of up to
    1024 terms over at most eight layers stay far below it; a wrong pooled row, weight or
    activation moves y by a large fraction of itself)."""
    from paper_2505_09142_amd.device import DeviceWeights
    from workloads import make_weights
    note(f"pool + head {shape.name}: {len(lens)} sequences")
    rng = np.random.default_rng(len(lens) + shape.d_model)
    b = pack([np.zeros(L, np.int32) for L in lens])
    T, d = b.total, shape.d_model
    hid = rng.standard_normal((T, d)).astype(np.float32)
    W = make_weights(dataclasses.replace(shape, n_layers=0), 77)
    head_keys = ("head_w1", "head_b1", "head_w2", "head_b2", "head_mid_w", "head_mid_b")
    dw = DeviceWeights(dataclasses.replace(shape, n_layers=0), {k: W.device[k] for k in head_keys if k in W.device})
    cfg = dw.cfg
    need = E.elis_pool_head_workspace_bytes(cfg, b.n, b.max_seqlen)
    buf, ws, wsb = workspace(need)
    d_hid, d_cu = dev(hid), dev(b.cu_seqlens)
    out = torch.full((b.n,), float("nan"), dtype=torch.float32, device="cuda")
    ok(E.elis_pool_head(dw.struct, d_hid.data_ptr(), d_cu.data_ptr(), b.n, T, b.max_seqlen, out.data_ptr(), ws, wsb,
                        stream()), "pool_head")
    st, bits = E.elis_read_status(ws, stream())
    assert st == E.ELIS_OK and bits == 0
    got = out.cpu().numpy().astype(np.float64)
    h64 = hid.astype(np.float64)
    ref = np.array([oracle.regression_head(oracle.pool(h64[b.cu_seqlens[s]:b.cu_seqlens[s + 1]], shape.pooling),
                                           W.master, shape) for s in range(b.n)])
    y, y_ref = (got - shape.out_shift) / shape.out_scale, (ref - shape.out_shift) / shape.out_scale
    err = np.abs(y - y_ref).max() / np.abs(y_ref).max()
    note(f"pool + head {shape.name}: max |y - y_ref| / max |y_ref| = {err:.3e}")
    assert err <= 1e-4
