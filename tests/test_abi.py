"""The C-ABI library on the host: it loads, exports every symbol the header
declares, and rejects invalid arguments with the documented status before
touching the device (no kernel is launched by any call here)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2505_09142_amd import _elis as E
from paper_2505_09142_amd.device import config_of
from workloads import BERT_BASE, TINY, TINY_HEAD8, XLMR_LARGE

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "elis.h")

FAKE = 0x1000  # never dereferenced: every call below fails validation first
FAKE_WS = 0x100000  # 256-byte aligned


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(elis_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(E.LIB_PATH):
        pytest.fail("libelis.so is not built (run python -m paper_2505_09142_amd.build)")
    return E.lib()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(E.SIGNATURES), "binding and header disagree"


def test_version_and_strings(lib):
    assert E.elis_abi_version() == 3
    for s in (0, -1, -2, -3, -4, -5, -6):
        assert E.elis_status_string(s).startswith("ELIS_")
    assert E.elis_status_string(123) == "unknown status"


def test_workspace_queries(lib):
    for shape in (TINY, BERT_BASE, XLMR_LARGE, TINY_HEAD8):
        cfg = config_of(shape)
        b = E.elis_predict_workspace_bytes(cfg, 1000, 8, 64)
        d, F = shape.d_model, shape.d_ff
        # fp32 residual + bf16 copy + qkv + attention out + fp32 pre-LN + FFN activation
        assert b >= 1000 * (4 * d + 2 * d + 6 * d + 2 * d + 4 * d + 2 * F)
        assert b % 256 == 0
        assert E.elis_predict_workspace_bytes(cfg, 7, 8, 64) == 0       # fewer tokens than sequences
        assert E.elis_predict_workspace_bytes(cfg, 100, 8, shape.max_pos + 1) == 0
    assert E.elis_select_workspace_bytes(0) == 0
    assert E.elis_select_workspace_bytes(E.elis_select_max_n() + 1) == 0
    assert E.elis_select_workspace_bytes(64) >= 4
    # above 8192 jobs: a tie list of up to n indices
    assert E.elis_select_workspace_bytes(8193) >= 4 * 8193
    assert E.elis_select_workspace_bytes(1 << 24) >= 4 * (1 << 24)
    assert E.elis_select_max_n() == 1 << 28
    assert E.elis_select_max_batch_cap(0) == 0
    assert E.elis_select_max_batch_cap(8192) == 2 ** 31 - 1
    assert E.elis_select_max_batch_cap(8193) == 8192
    assert E.elis_select_max_batch_cap(E.elis_select_max_n() + 1) == 0
    assert E.elis_attention_workspace_bytes(4, 100) > 0
    assert E.elis_attention_workspace_bytes(4, 3) == 0


def _weights(shape=TINY):
    cfg = config_of(shape)
    layers = (E.elis_layer_weights * max(1, shape.n_layers))()
    for l in range(shape.n_layers):
        for f, _ in E.elis_layer_weights._fields_:
            setattr(layers[l], f, FAKE)
    nmid = max(0, shape.n_head_layers - 2)
    mid = (ctypes.c_void_p * max(1, nmid))(*([FAKE] * nmid))
    midp = ctypes.cast(mid, ctypes.POINTER(ctypes.c_void_p)) if nmid else None
    w = E.elis_weights(cfg, FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.cast(layers, ctypes.POINTER(E.elis_layer_weights)),
                       FAKE, FAKE, FAKE, FAKE, midp, midp)
    w._keep = (layers, mid)
    return w


def _predict(w, ids=FAKE, cu=FAKE, n=4, T=100, max_seqlen=64, pred=FAKE, ws=FAKE_WS, wsb=1 << 40):
    return E.elis_predict_remaining(w, ids, cu, n, T, max_seqlen, pred, None, ws, wsb, None)


def test_predict_rejects_invalid_arguments(lib):
    w = _weights()
    assert _predict(None) == E.ELIS_EINVAL
    assert _predict(w, ids=None) == E.ELIS_EINVAL
    assert _predict(w, cu=None) == E.ELIS_EINVAL
    assert _predict(w, pred=None) == E.ELIS_EINVAL
    assert _predict(w, ws=None) == E.ELIS_EINVAL
    assert _predict(w, ws=FAKE_WS + 8) == E.ELIS_EINVAL          # misaligned workspace
    assert _predict(w, n=0) == E.ELIS_EINVAL
    assert _predict(w, n=-3) == E.ELIS_EINVAL
    assert _predict(w, T=0) == E.ELIS_EINVAL
    assert _predict(w, max_seqlen=TINY.max_pos + 1) == E.ELIS_ESHAPE
    assert _predict(w, max_seqlen=0) == E.ELIS_ESHAPE
    assert _predict(w, n=8, T=5) == E.ELIS_ESHAPE
    assert _predict(w, wsb=1000) == E.ELIS_EWORKSPACE


def test_predict_rejects_bad_config(lib):
    w = _weights()
    w.cfg.pooling = 7
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights()
    w.cfg.d_model = 96                                           # not a multiple of 64
    assert _predict(w) == E.ELIS_EUNSUPPORTED
    w = _weights()
    w.cfg.n_heads = 1                                            # d_head 128
    assert _predict(w) == E.ELIS_EUNSUPPORTED
    w = _weights()
    w.cfg.ln_eps = float("nan")
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights()
    w.layers[1].w_2 = None
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights()
    w.cfg.head_hidden = 16                                       # hidden width with a one-layer head
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights()
    w.cfg.head_hidden, w.cfg.head_layers = 16, 2
    w.head_w1 = None                                             # first layer missing
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights(TINY_HEAD8)
    w.head_mid_w = None                                          # middle layers missing
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights(TINY_HEAD8)
    w.cfg.head_act = 5
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights(TINY_HEAD8)
    w.cfg.head_layers = 0
    assert _predict(w) == E.ELIS_EINVAL
    w = _weights(TINY_HEAD8)
    w.cfg.head_hidden = 66                                       # not a multiple of 4
    assert _predict(w) == E.ELIS_EUNSUPPORTED


def test_select_rejects_invalid_arguments(lib):
    ok = dict(pred=FAKE, arr=FAKE, n=8, k=4, idx=FAKE, cnt=FAKE, ws=FAKE_WS, wsb=256)

    def call(**kw):
        a = {**ok, **kw}
        return E.elis_isrtf_select(a["pred"], a["arr"], a["n"], a["k"], a["idx"], a["cnt"], a["ws"], a["wsb"], None)

    assert call(pred=None) == E.ELIS_EINVAL
    assert call(arr=None) == E.ELIS_EINVAL
    assert call(cnt=None) == E.ELIS_EINVAL
    assert call(idx=None) == E.ELIS_EINVAL
    assert call(n=0) == E.ELIS_EINVAL
    assert call(k=-1) == E.ELIS_EINVAL
    assert call(ws=FAKE_WS + 4) == E.ELIS_EINVAL
    assert call(n=E.elis_select_max_n() + 1) == E.ELIS_ESHAPE
    assert call(wsb=0) == E.ELIS_EWORKSPACE
    # more than 8192 jobs: at most 8192 chosen
    big = E.elis_select_workspace_bytes(100000)
    assert call(n=100000, k=8193, wsb=big) == E.ELIS_EUNSUPPORTED
    assert call(n=100000, k=8192, wsb=big - 1) == E.ELIS_EWORKSPACE


def test_building_blocks_reject_invalid_arguments(lib):
    assert E.elis_linear(None, FAKE, FAKE, None, 4, 64, 64, 0, FAKE, None) == E.ELIS_EINVAL
    assert E.elis_linear(FAKE, FAKE, FAKE, None, 4, 64, 64, 2, FAKE, None) == E.ELIS_EINVAL  # residual missing
    assert E.elis_linear(FAKE, FAKE, FAKE, None, 4, 64, 64, 9, FAKE, None) == E.ELIS_EINVAL
    assert E.elis_linear(FAKE, FAKE, FAKE, None, 0, 64, 64, 0, FAKE, None) == E.ELIS_EINVAL
    assert E.elis_linear(FAKE, FAKE, FAKE, None, 4, 96, 64, 0, FAKE, None) == E.ELIS_EUNSUPPORTED
    assert E.elis_linear(FAKE, FAKE, FAKE, None, 4, 64, 80, 0, FAKE, None) == E.ELIS_EUNSUPPORTED
    assert E.elis_attention(FAKE, FAKE, 2, 10, 8, 2, 48, FAKE, FAKE_WS, 4096, None) == E.ELIS_EUNSUPPORTED
    assert E.elis_attention(FAKE, FAKE, 2, 1, 8, 2, 64, FAKE, FAKE_WS, 4096, None) == E.ELIS_ESHAPE
    assert E.elis_attention(FAKE, FAKE, 2, 10, 8, 2, 64, FAKE, FAKE_WS, 8, None) == E.ELIS_EWORKSPACE
    assert E.elis_attention(None, FAKE, 2, 10, 8, 2, 64, FAKE, FAKE_WS, 4096, None) == E.ELIS_EINVAL
    assert E.elis_layernorm(FAKE, FAKE, FAKE, 4, 64, 1e-5, None, None, None) == E.ELIS_EINVAL
    assert E.elis_layernorm(FAKE, FAKE, FAKE, 4, 100, 1e-5, FAKE, None, None) == E.ELIS_EUNSUPPORTED
    assert E.elis_layernorm(FAKE, FAKE, FAKE, 0, 64, 1e-5, FAKE, None, None) == E.ELIS_EINVAL


def test_linear_plan_host_only(lib):
    """The launch plan of a product is host arithmetic: rows split at a whole number of main-tile
    rows, the two launches cover [0, m), tiles of the shapes the library has, and the arguments
    elis_linear rejects are rejected here too."""
    tiles = {(64, 64), (64, 128), (128, 64), (128, 128), (256, 256)}
    rng = np.random.default_rng(5)
    splits = 0
    for _ in range(400):
        n = int(rng.choice([384, 512, 768, 1024, 2304, 3072, 4096, 320]))
        k = int(rng.choice([64, 128, 768, 1024, 3072, 4096]))
        m = int(rng.integers(1, 120000))
        epi = int(rng.integers(0, 3))
        st, (bm, bn, wg, m1, rbm, rbn, rwg) = E.elis_linear_plan(m, n, k, epi)
        assert st == E.ELIS_OK
        assert (bm, bn) in tiles and n % bn == 0 and wg in (1, 2, 4)
        assert 1 <= m1 <= m
        if m1 < m:
            splits += 1
            assert m1 % bm == 0 and (rbm, rbn) in tiles and n % rbn == 0 and rwg in (1, 2, 4)
            assert (rbm, rbn, rwg) != (bm, bn, wg)
            # the first launch fills whole rounds of work-group slots (256 CUs without a GPU): as
            # many whole rows of tiles as fit in the full rounds of a single launch
            per_row, slots = n // bn, wg * 256
            full = (-(-m // bm) * per_row) // slots * slots
            assert full >= slots and full - per_row < (m1 // bm) * per_row <= full
        else:
            assert (rbm, rbn, rwg) == (0, 0, 0)
    assert splits > 20
    assert E.elis_linear_plan(23931, 768, 3072, E.ELIS_EPI_BIAS_RES_F32)[1][3] < 23931
    assert E.elis_linear_plan(0, 768, 768, 0)[0] == E.ELIS_EINVAL
    assert E.elis_linear_plan(100, 100, 768, 0)[0] == E.ELIS_EUNSUPPORTED
    assert E.elis_linear_plan(100, 768, 100, 0)[0] == E.ELIS_EUNSUPPORTED
    assert E.elis_linear_plan(100, 768, 768, 3)[0] == E.ELIS_EINVAL


def test_linear_with_plan_rejects_invalid_plans(lib):
    FAKE = 256  # never dereferenced: every call below fails validation on the host
    def call(plan, m=1000, n=768, k=768, epi=E.ELIS_EPI_BIAS_BF16):
        return E.elis_linear_with_plan(FAKE, FAKE, FAKE, None, m, n, k, epi, plan, FAKE, None)
    assert call(None) == E.ELIS_EINVAL
    assert call((96, 128, 1, 1000, 0, 0, 0)) == E.ELIS_EINVAL        # unknown tile
    assert call((256, 256, 2, 1000, 0, 0, 0)) == E.ELIS_EINVAL       # 256 x 256 runs one per CU
    assert call((256, 256, 1, 1000, 0, 0, 0), n=640) == E.ELIS_EINVAL  # tile width must divide n
    assert call((128, 128, 2, 0, 0, 0, 0)) == E.ELIS_EINVAL          # m1 >= 1
    assert call((128, 128, 2, 1001, 0, 0, 0)) == E.ELIS_EINVAL       # m1 <= m
    assert call((128, 128, 2, 1000, 64, 128, 1)) == E.ELIS_EINVAL    # no rest when m1 == m
    assert call((128, 128, 2, 500, 64, 128, 1)) == E.ELIS_EINVAL     # m1 a multiple of main_bm
    assert call((128, 128, 2, 512, 128, 128, 2)) == E.ELIS_EINVAL    # rest differs from main
    assert call((128, 128, 2, 512, 0, 0, 0)) == E.ELIS_EINVAL        # rest missing
    assert call((128, 64, 2, 1000, 0, 0, 0)) == E.ELIS_EINVAL        # 128 x 64 only for n = 64 mod 128
    assert call((256, 256, 1, 512, 128, 64, 2), n=768) == E.ELIS_EINVAL
    assert call((128, 128, 2, 1000, 0, 0, 0), n=100) == E.ELIS_EUNSUPPORTED


def test_timing_api_host_only(lib):
    assert E.elis_timing_enable(0) == 0
    assert E.elis_timing_reset() == 0
    st, n, ms = E.elis_timing_read(0)
    assert st == 0 and n == 0 and ms == 0.0
    assert E.elis_timing_read(99)[0] == E.ELIS_EINVAL
    assert E.elis_timing_stride(0) == E.ELIS_EINVAL
    assert E.elis_timing_stride(-3) == E.ELIS_EINVAL
    assert E.elis_timing_stride(13) == 0
    assert E.elis_timing_stride(1) == 0


def test_job_table_rejects_invalid_arguments(lib):
    assert E.elis_jobs_table_bytes(0, 8) == 0
    assert E.elis_jobs_table_bytes(4, 1) == 0
    assert E.elis_jobs_table_bytes(100, 512) >= 100 * 511 * 4
    assert E.elis_jobs_select_workspace_bytes(0) == 0
    assert E.elis_jobs_select_workspace_bytes(100) >= 100 * (4 + 8 + 4)
    good = E.elis_job_table(FAKE_WS, 16, 8)
    assert E.elis_jobs_init(None, None) == E.ELIS_EINVAL
    assert E.elis_jobs_init(E.elis_job_table(None, 16, 8), None) == E.ELIS_EINVAL
    assert E.elis_jobs_init(E.elis_job_table(FAKE_WS + 4, 16, 8), None) == E.ELIS_EINVAL   # unaligned
    assert E.elis_jobs_init(E.elis_job_table(FAKE_WS, 0, 8), None) == E.ELIS_EINVAL
    assert E.elis_jobs_init(E.elis_job_table(FAKE_WS, 16, 1), None) == E.ELIS_EINVAL
    assert E.elis_jobs_start(good, None, FAKE, 2, None) == E.ELIS_EINVAL
    assert E.elis_jobs_start(good, FAKE, FAKE, -1, None) == E.ELIS_EINVAL
    assert E.elis_jobs_start(good, None, None, 0, None) == E.ELIS_OK                        # nothing to do
    assert E.elis_jobs_append(good, FAKE, FAKE, None, 2, 3, None) == E.ELIS_EINVAL           # tokens missing
    assert E.elis_jobs_append(good, FAKE, FAKE, FAKE, 2, -1, None) == E.ELIS_EINVAL
    assert E.elis_jobs_append(good, None, None, None, 0, 0, None) == E.ELIS_OK
    assert E.elis_jobs_pack(good, FAKE, 0, 4, 4, FAKE, FAKE, None) == E.ELIS_EINVAL
    assert E.elis_jobs_pack(good, FAKE, 2, 1, 4, FAKE, FAKE, None) == E.ELIS_ESHAPE          # fewer tokens than jobs
    assert E.elis_jobs_pack(good, FAKE, 2, 4, 9, FAKE, FAKE, None) == E.ELIS_ESHAPE          # max_seqlen > max_pos
    assert E.elis_jobs_store_pred(good, FAKE, None, 2, None) == E.ELIS_EINVAL
    ws = E.elis_jobs_select_workspace_bytes(100)
    assert E.elis_jobs_select(good, FAKE, 100, 4, FAKE, FAKE, FAKE_WS, ws - 1, None) == E.ELIS_EWORKSPACE
    assert E.elis_jobs_select(good, FAKE, 0, 4, FAKE, FAKE, FAKE_WS, ws, None) == E.ELIS_EINVAL
    assert E.elis_jobs_select(good, FAKE, 100, -1, FAKE, FAKE, FAKE_WS, ws, None) == E.ELIS_EINVAL
    big = E.elis_jobs_select_workspace_bytes(10000)
    assert E.elis_jobs_select(good, FAKE, 10000, 9000, FAKE, FAKE, FAKE_WS, big, None) == E.ELIS_EUNSUPPORTED
    # aged select: same checks plus a missing wait array or a non-finite aging rate
    assert E.elis_jobs_select_aged(good, FAKE, None, 1.0, 100, 4, FAKE, FAKE, FAKE_WS, ws, None) == E.ELIS_EINVAL
    assert E.elis_jobs_select_aged(good, FAKE, FAKE, float("nan"), 100, 4, FAKE, FAKE, FAKE_WS, ws, None) == E.ELIS_EINVAL
    assert E.elis_jobs_select_aged(good, FAKE, FAKE, float("inf"), 100, 4, FAKE, FAKE, FAKE_WS, ws, None) == E.ELIS_EINVAL
    assert E.elis_jobs_select_aged(good, FAKE, FAKE, 1.0, 100, 4, FAKE, FAKE, FAKE_WS, ws - 1, None) == E.ELIS_EWORKSPACE
    assert E.elis_jobs_select_aged(good, FAKE, FAKE, 1.0, 0, 4, FAKE, FAKE, FAKE_WS, ws, None) == E.ELIS_EINVAL
    assert E.elis_jobs_select_aged(good, FAKE, FAKE, 1.0, 10000, 9000, FAKE, FAKE, FAKE_WS, big, None) == \
        E.ELIS_EUNSUPPORTED


def test_pool_head_rejects_invalid_arguments(lib):
    def call(w, hid=FAKE, cu=FAKE, n=4, T=100, msl=64, pred=FAKE, ws=FAKE_WS, wsb=1 << 30):
        return E.elis_pool_head(w, hid, cu, n, T, msl, pred, ws, wsb, None)

    w = _weights(TINY_HEAD8)
    cfg = config_of(TINY_HEAD8)
    need = E.elis_pool_head_workspace_bytes(cfg, 4, 64)
    assert need > 0 and need % 256 == 0
    # mean pooling: a partial sum per 64-row chunk of every sequence (one chunk at 64 tokens), the
    # pooled rows and two hidden buffers
    d, hh = TINY_HEAD8.d_model, TINY_HEAD8.head_hidden
    assert need >= 4 * 1 * d * 4 + 4 * d * 4 + 2 * 4 * hh * 4
    assert E.elis_pool_head_workspace_bytes(cfg, 4, 128) >= need + 4 * d * 4
    assert E.elis_pool_head_workspace_bytes(cfg, 0, 64) == 0
    assert E.elis_pool_head_workspace_bytes(cfg, 4, TINY_HEAD8.max_pos + 1) == 0
    assert call(None) == E.ELIS_EINVAL
    assert call(w, hid=None) == E.ELIS_EINVAL
    assert call(w, cu=None) == E.ELIS_EINVAL
    assert call(w, pred=None) == E.ELIS_EINVAL
    assert call(w, ws=FAKE_WS + 16) == E.ELIS_EINVAL
    assert call(w, n=0) == E.ELIS_EINVAL
    assert call(w, n=8, T=5) == E.ELIS_ESHAPE
    assert call(w, msl=TINY_HEAD8.max_pos + 1) == E.ELIS_ESHAPE
    assert call(w, wsb=need - 1) == E.ELIS_EWORKSPACE
    w.head_mid_b = None
    assert call(w) == E.ELIS_EINVAL
    # only the head's pointers are read: encoder pointers may be missing
    w = _weights(TINY_HEAD8)
    w.word = None
    w.layers = None
    assert call(w, wsb=need - 1) == E.ELIS_EWORKSPACE


def test_select_noalloc_limits_and_rejections(lib):
    """The allocation-free select's fixed scratch holds the workspace of its largest n; every
    invalid call is refused on the host (no device work)."""
    nmax = E.ELIS_SELECT_NOALLOC_MAX_N
    assert E.elis_select_workspace_bytes(nmax) <= E.ELIS_SELECT_NOALLOC_SCRATCH_BYTES
    hdr = open(HEADER).read()
    assert f"#define ELIS_SELECT_NOALLOC_MAX_N (1 << {nmax.bit_length() - 1})" in hdr
    assert "#define ELIS_SELECT_NOALLOC_SCRATCH_BYTES (3u << 20)" in hdr

    def call(pred=FAKE, arr=FAKE, n=8, k=4, idx=FAKE, cnt=FAKE):
        return E.elis_isrtf_select_noalloc(pred, arr, n, k, idx, cnt, None)

    assert call(pred=None) == E.ELIS_EINVAL
    assert call(arr=None) == E.ELIS_EINVAL
    assert call(cnt=None) == E.ELIS_EINVAL
    assert call(idx=None) == E.ELIS_EINVAL
    assert call(n=0) == E.ELIS_EINVAL
    assert call(k=-1) == E.ELIS_EINVAL
    assert call(n=nmax + 1) == E.ELIS_ESHAPE
    assert call(n=nmax, k=8193) == E.ELIS_EUNSUPPORTED
