"""Host mirrors of two pieces of the attention path's index arithmetic (CPU only).

1. The seq-map kernel's attention work list (seqmap.hip): a counting sort of the
   query tiles on each sequence's number of 64-key tiles (capped at 64), longest
   first, batch order inside a bucket, built per 1024-thread chunk from in-wave
   ranks, per-wave bucket totals and per-bucket carries; the slots between the
   count and the capacity get length 0. Checked: the entries written are a
   bijection onto [0, min(count, capacity)), every write lies below the capacity
   the workspace holds (the attention grid's size, so every work-group reads a
   written slot), the order is longest first and stable, and each entry names the
   right (sequence, query tile).
2. The d_head-64 V tile (attention.hip): direct-to-LDS loads place row R's
   logical 16-byte chunk c at physical chunk c ^ (2 * ((R >> 1) & 3)); the PV
   operand is read with ds_read_b64_tr_b16, whose result for lane i of a 16-lane
   group is element i % 4 of the 8-byte units addressed by lanes 4r + i // 4,
   r = 0..3 (the layout of the instruction). Checked: every LDS access stays in
   the tile's buffer, the transposed reads hand lane l of the wave exactly
   V[32 kc + 4 (l // 16) + r (+16)][16 dt + l % 16], the keys of the P^T operand
   slots, and the 32 lanes of each half-wave touch 64 distinct banks.
"""
import numpy as np
import pytest

KT, KW, KB, RPB = 1024, 64, 64, 128


def bucket(L):
    t = (L + 63) // 64
    return t - 1 if t < KB else KB - 1


def capacity(n, total):
    return (total + RPB - 1) // RPB + n


def build_work_list(lens, cap):
    """The kernel's construction, thread by thread; returns {index: (s, q)}."""
    n = len(lens)
    tiles = [(L + RPB - 1) // RPB for L in lens]
    hist = [0] * KB
    for L, t in zip(lens, tiles):
        hist[bucket(L)] += t
    # Wave 0: lane l scans bucket KB-1-l (inclusive scan minus own count).
    base = [0] * KB
    run = 0
    for lane in range(KB):
        b = KB - 1 - lane
        base[b] = run
        run += hist[b]
    carry = [0] * KB
    work = {}
    for cb in range(0, n, KT):
        wave_b = np.zeros((KT // KW, KB), dtype=np.int64)
        first = {}
        for w in range(KT // KW):
            ids = [cb + w * KW + lane for lane in range(KW)]
            bs = [bucket(lens[s]) if s < n else -1 for s in ids]
            ts = [tiles[s] if s < n else 0 for s in ids]
            nv = max(0, min(KW, n - cb - w * KW))
            for lane in range(KW):
                off = sum(ts[o] for o in range(nv) if o < lane and bs[o] == bs[lane])
                wave_b[w, lane] = sum(ts[o] for o in range(nv) if bs[o] == lane)
                first[ids[lane]] = off
        for w in range(KT // KW):
            for lane in range(KW):
                s = cb + w * KW + lane
                if s >= n:
                    continue
                b = bucket(lens[s])
                f = base[b] + carry[b] + first[s] + int(wave_b[:w, b].sum())
                for q in range(tiles[s]):
                    idx = f + q
                    if idx < cap:
                        assert idx not in work, "two entries written to one slot"
                        work[idx] = (s, q)
        for b in range(KB):
            carry[b] += int(wave_b[:, b].sum())
    for idx in range(sum(tiles), cap):  # slots past the list's end: length 0, the work-group exits
        assert idx not in work
        work[idx] = None
    return work, sum(tiles)


def check_list(lens, total):
    cap = capacity(len(lens), total)
    work, count = build_work_list(lens, cap)
    m = min(count, cap)
    assert sorted(work) == list(range(cap))  # every slot of the grid reads a written entry
    assert all(work[i] is None for i in range(m, cap)) and all(work[i] is not None for i in range(m))
    keys = [(-bucket(lens[work[i][0]]), work[i][0], work[i][1]) for i in range(m)]
    assert keys == sorted(keys), "not longest first, batch order within a bucket"
    if count <= cap:  # every query tile of every sequence listed once
        assert sorted(work[i] for i in range(m)) == sorted((s, q) for s, L in enumerate(lens) for q in range((L + RPB - 1) // RPB))
    return count, cap


@pytest.mark.parametrize("seed", range(6))
def test_work_list_random_batches(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 2600))
    hi = int(rng.choice([130, 520, 2048, 9000]))
    lens = [int(x) for x in rng.integers(1, hi, n)]
    count, cap = check_list(lens, sum(lens))
    assert count <= cap


def test_work_list_edge_batches():
    check_list([1], 1)
    check_list([1] * 3000, 3000)              # three chunks, every sequence one tile
    check_list([128, 129, 64, 65, 4096, 4097, 8192], 128 + 129 + 64 + 65 + 4096 + 4097 + 8192)
    check_list([512] * 64, 512 * 64)          # one bucket only
    check_list(list(range(1, 1500)), sum(range(1, 1500)))


def test_work_list_over_capacity_is_clipped():
    # Malformed boundaries can give clamped lengths whose tiles exceed the capacity:
    # entries past it are dropped and no write leaves the list.
    lens = [9000, 7, 1]
    cap = 10
    work, count = build_work_list(lens, cap)
    assert count > cap and sorted(work) == list(range(cap)) and None not in work.values()


def test_v_tile_direct_load_and_transposed_read():
    DH, BKV, WAVES = 64, 64, 4
    cpr, krl = DH // 8, KW // (DH // 8)
    klw = 16 // krl
    vbuf = BKV * DH  # bf16 elements per buffer
    # Direct-to-LDS loads: wave w, load i, lane j writes 8 elements at w*16*DH + i*krl*DH + 8 j.
    lds = np.full(vbuf, -1, dtype=np.int64)  # holds key * 1000 + d
    for w in range(WAVES):
        for i in range(klw):
            for j in range(KW):
                row = w * 16 + i * krl + j // cpr
                vswz = ((row >> 1) & 3) << 2
                chunk = (j % cpr) ^ (vswz >> 1)  # logical source chunk
                dst = w * 16 * DH + i * krl * DH + 8 * j
                assert 0 <= dst and dst + 8 <= vbuf
                assert lds[dst:dst + 8].max() == -1, "element written twice"
                lds[dst:dst + 8] = [row * 1000 + chunk * 8 + e for e in range(8)]
    assert lds.min() >= 0
    for kc in range(2):
        for dt in range(DH // 16):
            addr = np.zeros((KW, 2), dtype=np.int64)
            for lane in range(KW):
                g, j16 = lane // 16, lane % 16
                r, q = j16 >> 2, j16 & 3
                row = kc * 32 + 4 * g + r
                p0 = row * DH + (4 * (dt ^ ((row >> 1) & 3)) + q) * 4
                # The kernel forms the lane part once (key row 4 g + r) and adds 32 kc rows:
                # the swizzle reads bits 1-2 of the row, which 32 kc leaves alone.
                r0 = 4 * g + r
                assert p0 == r0 * DH + (4 * (dt ^ ((r0 >> 1) & 3)) + q) * 4 + kc * 32 * DH
                for h, p in enumerate((p0, p0 + 16 * DH)):
                    assert 0 <= p and p + 4 <= vbuf
                    addr[lane, h] = p
            for h in range(2):
                for lane in range(KW):
                    grp = lane // 16 * 16
                    i = lane % 16
                    got = [lds[addr[grp + 4 * r + i // 4, h] + i % 4] for r in range(4)]
                    g = lane // 16
                    want = [(kc * 32 + 16 * h + 4 * g + r) * 1000 + dt * 16 + i for r in range(4)]
                    assert got == want
                for half in range(2):
                    bset = set()
                    for lane in range(32 * half, 32 * half + 32):
                        w0 = addr[lane, h] * 2 // 4  # first 4-byte word of the 8-byte unit
                        bset.update({w0 % 64, (w0 + 1) % 64})
                    assert len(bset) == 64, "bank conflict in a transposed read"
