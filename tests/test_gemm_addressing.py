"""Host mirror of the GEMM kernels' address arithmetic (CPU only, no GPU).

Every index expression of gemm.hip that forms a global or LDS address is
re-evaluated here, in numpy over all work-groups, waves and lanes of a launch,
for every tile configuration the launch plans can route to and for the plans
the library picks (elis_linear_plan, a host-only call) over the encoder shapes
at the sizes the plan sweep times. The checks:

* the work-group -> tile map (XCD remap, then GROUP_M grouping) is a bijection
  onto the tile grid;
* every global read (activation rows clamped at the ragged end, weight rows,
  bias, residual, LayerNorm parameters and row statistics) stays inside its
  buffer; every global store stays inside the output and covers each output
  element exactly once;
* every direct-to-LDS load and every fragment read stays inside its stage and
  operand region, each stage is filled exactly once per k-slab, and the XOR
  swizzle makes a fragment read of (row, logical chunk) see the global chunk it
  names;
* the epilogue's LDS staging (writes and read-back) stays inside the stage
  buffers and inside the wave's own rows;
* a two-launch plan's second launch (row offset m1) addresses only rows
  [m1, M) of the full buffers.

The configuration list is read from gemm.hip itself (the launch_gemm_config
switch and kTileShapes), so a configuration added there without a mirror here
fails the first test.
"""
import os
import re

import numpy as np
import pytest

from paper_2505_09142_amd import _elis as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GEMM_SRC = os.path.join(ROOT, "paper_2505_09142_amd", "csrc", "gemm.hip")
WAVE = 64
BK = 64
GROUP_M = 8

# id -> (kind, BM, BN, WM, WN, MI, OCC, S); kind "sched" = gemm_sched_kernel, "reg" = gemm_kernel
CONFIGS = {
    1: ("reg", 128, 64, 2, 2, 16, 2, 2),
    21: ("sched", 256, 256, 2, 4, 32, 1, 2),
    32: ("sched", 128, 128, 2, 2, 32, 2, 2),
    33: ("sched", 64, 128, 2, 2, 32, 2, 2),
    34: ("sched", 64, 128, 2, 2, 32, 1, 4),
    35: ("sched", 64, 64, 2, 2, 32, 4, 2),
    36: ("sched", 64, 64, 2, 2, 32, 2, 4),
}
EPIS = (E.ELIS_EPI_BIAS_BF16, E.ELIS_EPI_BIAS_GELU_BF16, E.ELIS_EPI_BIAS_RES_F32)
TILE_TO_CFG = {(v[1], v[2], v[6]): c for c, v in CONFIGS.items()}  # (bm, bn, work-groups per CU) -> id


def test_mirror_covers_every_configuration():
    src = open(GEMM_SRC).read()
    found = {}
    for cid, kind, args in re.findall(r"case (\d+): return launch_(sched|tile)<([^>]*)>", src):
        v = [int(x) for x in args.split(",")]
        bm, bn, wm, wn, mi = v[:5]
        if kind == "sched":
            occ = v[5] if len(v) > 5 else 1
            s = v[6] if len(v) > 6 else 2
            found[int(cid)] = ("sched", bm, bn, wm, wn, mi, occ, s)
        else:
            found[int(cid)] = ("reg", bm, bn, wm, wn, mi, 2, 2)
    assert found == CONFIGS
    shapes = re.search(r"kTileShapes\[\] = \{(.*?)\};", src, re.S).group(1)
    listed = {int(c): (int(bm), int(bn), int(o)) for c, bm, bn, o in
              re.findall(r"\{(\d+), (\d+), (\d+), (\d+)\}", shapes)}
    assert listed == {c: (v[1], v[2], v[6]) for c, v in CONFIGS.items()}
    # the slab depth is fixed: no other depth is left in the template
    assert "constexpr int kBK = 64;" in src and not re.search(r"template <[^>]*\bint BK\b", src)


# ----------------------------------------------------------------------------- tile map

def xcd_remap(bid, nblk):
    per, rem = nblk // 8, nblk % 8
    xcd, local = bid % 8, bid // 8
    return xcd * per + np.minimum(xcd, rem) + local


def grouped_tile(t, tiles_m, tiles_n, gm):
    per_group = gm * tiles_n
    g = t // per_group
    first = g * gm
    rows = np.minimum(tiles_m - first, gm)
    r = t - g * per_group
    return first + r % rows, r // rows


def tile_map(kind, M, N, BM, BN):
    tiles_m, tiles_n = -(-M // BM), N // BN
    nblk = tiles_m * tiles_n
    bid = np.arange(nblk)
    t = xcd_remap(bid, nblk)
    if kind == "sched":
        tm, tn = grouped_tile(t, tiles_m, tiles_n, GROUP_M)
    else:
        tm, tn = t // tiles_n, t % tiles_n
    return tm, tn, tiles_m, tiles_n


@pytest.mark.parametrize("nblk", list(range(1, 70)) + [255, 256, 257, 1000, 4320])
def test_xcd_remap_is_a_bijection(nblk):
    assert np.array_equal(np.sort(xcd_remap(np.arange(nblk), nblk)), np.arange(nblk))


@pytest.mark.parametrize("tiles_m,tiles_n", [(1, 1), (3, 12), (8, 3), (9, 3), (17, 12), (361, 12), (95, 1)])
def test_grouped_tile_is_a_bijection(tiles_m, tiles_n):
    tm, tn = grouped_tile(np.arange(tiles_m * tiles_n), tiles_m, tiles_n, GROUP_M)
    assert tm.min() >= 0 and tm.max() < tiles_m and tn.min() >= 0 and tn.max() < tiles_n
    assert len(set(zip(tm.tolist(), tn.tolist()))) == tiles_m * tiles_n


def corner_tiles(tm, tn, tiles_m, tiles_n, full_cover):
    """Every tile for the exact-cover checks; else the tiles in the first and last tile row and
    column. Every address below grows with the tile's first row and column (the clamps and the
    store guard included), so those tiles hold each address's extremes."""
    if full_cover:
        return tm, tn
    keep = ((tm == 0) | (tm == tiles_m - 1)) & ((tn == 0) | (tn == tiles_n - 1))
    return tm[keep], tn[keep]


# ----------------------------------------------------------------------------- scheduled kernel

def sw(row):
    return (row >> 1) & 7


def check_sched(M, N, K, epi, cfg, full_cover):
    """gemm_sched_kernel<BM, BN, WM, WN, 32, EPI, OCC, S> on an M x N x K product."""
    _, BM, BN, WM, WN, MI, OCC, S = cfg
    NW = WM * WN
    TM, TN = BM // WM, BN // WN
    FM, FN = TM // MI, TN // MI
    CPR = BK // 8
    RPI = WAVE // CPR
    LA, LB = BM // RPI // NW, BN // RPI // NW
    assert BM % (RPI * NW) == 0 and BN % (RPI * NW) == 0
    STAGE = (BM + BN) * BK          # uint16 elements
    SMEM = S * STAGE
    NGL = LA + LB
    assert S * NGL < 64             # the vmcnt field holds every outstanding load
    KT = K // BK
    KS = BK // 16                   # 32 x 32 x 16 k-steps per slab
    GROUPS = WAVE // MI
    assert KS % 2 == 0

    tm, tn, tiles_m, tiles_n = tile_map("sched", M, N, BM, BN)
    assert np.array_equal(np.sort(tm * tiles_n + tn), np.arange(tiles_m * tiles_n))
    tm, tn = corner_tiles(tm, tn, tiles_m, tiles_n, full_cover)
    m0, n0 = tm * BM, tn * BN                      # [tiles]
    wid = np.arange(NW)[:, None]
    lane = np.arange(WAVE)[None, :]
    wm, wn = wid // WN, wid % WN

    # --- direct-to-LDS loads: lane i's 16 bytes land at the wave's LDS base + 8 * i elements
    for which, L, rows_of, base in (("A", LA, BM, 0), ("B", LB, BN, BM * BK)):
        cover = np.zeros(STAGE, np.int64)
        for i in range(L):
            row = (wid * L + i) * RPI + lane // CPR                   # [NW, 64]
            c = (lane % CPR) ^ sw(row)
            assert row.max() < rows_of
            dst = base + (wid * L + i) * RPI * BK + 8 * lane          # element offset in the stage
            assert dst.min() >= base and dst.max() + 8 <= base + rows_of * BK
            # the lane's LDS chunk (row, p) holds logical chunk p ^ sw(row)
            p = (dst - base - row * BK) // 8
            assert np.array_equal(p ^ sw(row), c)
            for e in range(8):
                np.add.at(cover, (dst + e).ravel(), 1)
            if which == "A":
                gr = np.minimum(m0[:, None, None] + row[None], M - 1)  # ragged tail: re-read the last row
                src_lo = gr * K + c * 8                               # at k0 = 0
                src_hi = gr * K + c * 8 + (KT - 1) * BK + 8           # at the last slab
                assert src_lo.min() >= 0 and src_hi.max() <= M * K
            else:
                gr = n0[:, None, None] + row[None]
                assert gr.max() < N
                src_hi = gr * K + c * 8 + (KT - 1) * BK + 8
                assert src_hi.max() <= N * K
        region = cover[base:base + rows_of * BK]
        assert np.all(region == 1), f"{which} region of a stage filled unevenly"
    # stages: slab kt goes to stage kt % S at offset (kt % S) * STAGE
    assert (S - 1) * STAGE + STAGE <= SMEM

    # --- fragment reads: rows wm*TM + i*32 + rl (A) / BM + wn*TN + j*32 + rl (B), chunk (ks*2+kg)^sw(rl)
    rl, kg = lane % MI, lane // MI
    rs = sw(rl)
    for ks in range(KS):
        c = ((ks * GROUPS + kg) ^ rs) * 8
        for i in range(FM):
            row = wm * TM + i * MI + rl
            assert np.array_equal(sw(row), rs + 0 * row)                 # fragment rows start at multiples of 32
            off = row * BK + c
            assert off.min() >= 0 and off.max() + 8 <= BM * BK
            # reading physical chunk c/8 of `row` yields logical chunk (c/8) ^ sw(row) = ks*2 + kg
            assert np.array_equal(((off - row * BK) // 8) ^ sw(row), ks * GROUPS + kg + 0 * row)
        for j in range(FN):
            row = wn * TN + j * MI + rl
            off = BM * BK + row * BK + c
            assert off.min() >= BM * BK and off.max() + 8 <= STAGE

    # --- epilogue staging through LDS
    f32 = epi == E.ELIS_EPI_BIAS_RES_F32
    EB = 4 if f32 else 2
    ROWB = TN * EB
    PITCH = ROWB + 16
    LPR = ROWB // 16
    RPR = WAVE // LPR
    NRR = 32 // RPR
    assert NW * 32 * PITCH <= SMEM * 2
    stg = wid * 32 * PITCH                                           # bytes
    for j in range(FN):
        for q in range(4):
            col = j * MI + 8 * q + 4 * kg
            w0 = stg + rl * PITCH + col * EB
            assert w0.min() >= 0 and (w0 + 4 * EB).max() <= SMEM * 2
            assert ((w0 + 4 * EB) <= stg + 32 * PITCH).all() and (col * EB + 4 * EB <= ROWB).all()
            bias_hi = n0[:, None, None] + wn[None] * TN + col[None] + 4
            assert bias_hi.max() <= N
    ch = lane % LPR
    nl = n0[:, None, None] + wn[None] * TN + ch[None] * (16 // EB)    # [tiles, NW, 64]
    assert (nl + 16 // EB).max() <= N
    if f32:
        assert (nl + 4).max() <= N                                   # LayerNorm g, b of those columns
    written = np.zeros(M * N, np.int32) if full_cover else None
    for i in range(FM):
        for rr in range(NRR):
            row = rr * RPR + lane // LPR
            rd = stg + row * PITCH + ch * 16
            assert row.max() < 32 and (rd + 16).max() <= SMEM * 2 and ((rd + 16) <= stg + 32 * PITCH).all()
            m = m0[:, None, None] + wm[None] * TM + i * MI + row[None]
            mc = np.minimum(m, M - 1)                                 # residual / stats rows: clamped
            if f32:
                assert (mc * N + nl + 4).max() <= M * N and mc.min() >= 0
            keep = m < M                                              # rows past the end store nothing
            o = m * N + nl
            assert not keep.any() or (o[keep].min() >= 0 and (o[keep] + 16 // EB).max() <= M * N)
            if written is not None:
                for e in range(16 // EB):
                    np.add.at(written, (o[keep] + e).ravel(), 1)
    if written is not None:
        assert np.all(written == 1), "each output element is stored exactly once"


def check_reg(M, N, K, epi, cfg, full_cover):
    """gemm_kernel<128, 64, 2, 2, 16, EPI>: register-staged slabs, 16 x 16 x 32 blocks."""
    _, BM, BN, WM, WN, MI, _, _ = cfg
    NT = WM * WN * WAVE
    TM, TN = BM // WM, BN // WN
    FM, FN = TM // MI, TN // MI
    ACH, BCH = BM * 8 // NT, BN * 8 // NT
    KT = K // BK
    tm, tn, tiles_m, tiles_n = tile_map("reg", M, N, BM, BN)
    assert np.array_equal(np.sort(tm * tiles_n + tn), np.arange(tiles_m * tiles_n))
    tm, tn = corner_tiles(tm, tn, tiles_m, tiles_n, full_cover)
    m0, n0 = tm * BM, tn * BN
    tid = np.arange(NT)
    for CH, rows_of, which in ((ACH, BM, "A"), (BCH, BN, "B")):
        cover = np.zeros(rows_of * BK, np.int64)
        for i in range(CH):
            ident = tid + i * NT
            row, c = ident >> 3, ident & 7
            assert row.max() < rows_of
            l = row * BK + ((c ^ (row & 7)) * 8)
            for e in range(8):
                np.add.at(cover, l + e, 1)
            if which == "A":
                gr = np.minimum(m0[:, None] + row[None], M - 1)
                assert (gr * K + c * 8 + (KT - 1) * BK + 8).max() <= M * K
            else:
                gr = n0[:, None] + row[None]
                assert gr.max() < N and (gr * K + c * 8 + (KT - 1) * BK + 8).max() <= N * K
        assert np.all(cover == 1)
    lane = tid % WAVE
    wid = tid // WAVE
    wm, wn = wid // WN, wid % WN
    rl, kg = lane % MI, lane // MI
    for ks in range(BK // 32):
        c = ks * (WAVE // MI) + kg
        for i in range(FM):
            row = wm * TM + i * MI + rl
            assert (row * BK + ((c ^ (row & 7)) * 8) + 8).max() <= BM * BK
        for j in range(FN):
            row = wn * TN + j * MI + rl
            assert (row * BK + ((c ^ (row & 7)) * 8) + 8).max() <= BN * BK
    written = np.zeros(M * N, np.int32) if full_cover else None
    for i in range(FM):
        m = m0[:, None] + wm[None] * TM + i * MI + rl[None]
        keep = m < M
        for j in range(FN):
            n = n0[:, None] + wn[None] * TN + j * MI + 4 * kg[None]
            assert (n + 4).max() <= N
            o = m * N + n
            assert not keep.any() or (o[keep] + 4).max() <= M * N
            if written is not None:
                for e in range(4):
                    np.add.at(written, (o[keep] + e).ravel(), 1)
    if written is not None:
        assert np.all(written == 1)


def check_config(cid, M, N, K, epi, full_cover):
    cfg = CONFIGS[cid]
    assert N % cfg[2] == 0 and K % BK == 0
    (check_sched if cfg[0] == "sched" else check_reg)(M, N, K, epi, cfg, full_cover)


SMALL_M = [1, 2, 31, 32, 33, 63, 64, 65, 127, 129, 255, 256, 257, 300, 511, 513]


@pytest.mark.parametrize("cid", sorted(CONFIGS))
@pytest.mark.parametrize("epi", EPIS)
def test_every_configuration_small_sizes_exact_cover(cid, epi):
    bn = CONFIGS[cid][2]
    N = 192 if cid == 1 else 2 * max(bn, 128)
    for M in SMALL_M:
        check_config(cid, M, N, 128, epi, full_cover=True)


# The plan sweep's sizes: M = 1K .. 92K for the encoder shapes (N, K) of BERT-base and XLM-R-large.
SWEEP_M = sorted(set([1024, 1536, 2048, 2500, 3000, 4096, 6000, 8192, 12000, 16384, 20000, 23931, 24576, 30000,
                      32768, 40000, 45000, 49152, 55000, 60000, 65536, 70000, 75000, 80000, 85000, 88000, 90000,
                      92160, 92233, 93000, 100718, 109400]))
SHAPES = [(2304, 768), (768, 768), (3072, 768), (768, 3072), (3072, 1024), (1024, 1024), (4096, 1024),
          (1024, 4096)]


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(E.LIB_PATH):
        pytest.fail("libelis.so is not built (run python -m paper_2505_09142_amd.build)")
    return E.lib()


@pytest.mark.parametrize("n,k", SHAPES)
def test_chosen_plans_stay_in_bounds(lib, n, k):
    checked = 0
    for epi in EPIS:
        for M in SWEEP_M:
            st, plan = E.elis_linear_plan(M, n, k, epi)
            assert st == E.ELIS_OK
            main = TILE_TO_CFG[(plan[0], plan[1], plan[2])]
            m1 = plan[3]
            assert 1 <= m1 <= M
            check_config(main, m1, n, k, epi, full_cover=False)
            if m1 < M:
                assert m1 % plan[0] == 0
                rest = TILE_TO_CFG[(plan[4], plan[5], plan[6])]
                # second launch: operands offset by m1 rows, M - m1 rows of its own
                check_config(rest, M - m1, n, k, epi, full_cover=False)
                assert m1 + (M - m1) == M
            checked += 1
    assert checked == len(EPIS) * len(SWEEP_M)


@pytest.mark.parametrize("cid", [21, 32, 33, 34, 35, 36])
def test_each_configuration_at_the_largest_sizes(cid):
    """The large tiles at the largest token counts; the 64-row tiles (planned over at most four rounds
    of 256 compute units) at the largest M that fits in four rounds, and one row of tiles past it."""
    _, bm, bn, _, _, _, occ, _ = CONFIGS[cid]
    for n, k in SHAPES:
        if n % bn:
            continue
        if bm >= 128:
            sizes = (92233, 109400)
        else:
            m4 = 4 * occ * 256 // (n // bn) * bm
            sizes = (m4, m4 + 1)
        for M in sizes:
            check_config(cid, M, n, k, E.ELIS_EPI_BIAS_RES_F32, full_cover=False)
