// Variable-length bidirectional multi-head attention over a packed batch
// (the encoder's self-attention: every token of a sequence attends to every
// token of the same sequence, and to nothing else).
//
// Work decomposition. A work-group takes one (sequence, head, 128-query tile);
// the tile table built by the seq-map kernel maps blockIdx.x to its sequence.
// Each of the 4 waves owns 32 queries (two 16-query MFMA blocks) and streams
// the sequence's keys and values through LDS in 64-token tiles, keeping a
// running maximum and running sum per query (online softmax), so the score
// matrix never leaves registers.
//
// Transposed formulation. The scores are computed as S^T = K Q^T and the
// output as O^T = V^T P^T on v_mfma_f32_16x16x32_bf16. With that order every
// lane holds, for ONE query (its lane % 16), four consecutive keys of each
// 16-key block in the accumulator layout; those accumulators, rounded to bf16,
// are directly the lane's slice of the P^T operand of the second product (the
// 8 k-slots of lane group g are keys {4g..4g+3} and {16+4g..16+4g+3} of a
// 32-key chunk). The row maximum of a query is therefore a reduction over the
// lane's own registers plus two lane-pair exchanges (v_permlane16_swap and
// v_permlane32_swap: lanes l, l^16, l^32, l^48 share a query). The row sum
// comes from the matrix cores: one extra 16-row block of O^T whose V^T rows are
// all ones accumulates sum_k P[q][k] over the same bf16 P that multiplies V, so
// the output is normalised by exactly the weights it was built from.
//
// LDS. K is stored row-major with 16-byte chunks XOR-swizzled by row pairs
// (the 16 rows one fragment read touches then cover every bank once). With d_head 64,
// V is stored row-major too, its 8-byte units XOR-swizzled by row pairs, and the
// V^T operand is read with ds_read_b64_tr_b16, which transposes 4x4 blocks of bf16
// across the lanes of a 16-lane group; both tiles go from HBM straight into LDS with
// no register staging. With d_head 32, V is staged through registers and stored
// transposed (V^T[d][key], rows padded to 72 keys, keys permuted within each 32-key
// chunk, see vt_pos) so that a lane's 8 keys for one d are one 16-byte read. Two LDS
// buffers: the next tile is in flight while the current one is multiplied, so each
// tile costs one barrier and its load latency is hidden.
#include <math.h>

#include "kernels.h"

namespace elis {

namespace {

constexpr int kWaves = 4;
constexpr int kQPerWave = 32;
constexpr int kBQ = kWaves * kQPerWave;  // == kAttnRowsPerBlock
constexpr int kBKV = 64;
constexpr int kVtStride = kBKV + 8;
static_assert(kBQ == kAttnRowsPerBlock, "tile table and kernel must agree");

template <int DH>
__device__ __forceinline__ int kswz(int row) {
    // chunks per K row: DH/8 (8 for d_head 64, 4 for 32). A 16-row fragment read with 16 bytes
    // per lane is conflict-free when (bank group of the row start, chunk) is distinct over the
    // 16 rows: rows start on 2 (d_head 64) or 4 (d_head 32) bank groups.
    constexpr int CPR = DH / 8;
    return CPR == 8 ? ((row >> 1) & 7) : ((row >> 2) & 3);
}

// Position of key k in a V^T row. The P^T operand of lane group g holds keys {4g..4g+3} and
// {16+4g..16+4g+3} of each 32-key chunk (the accumulator layout of S^T); storing key
// 32c + 16h + 4g + r at 32c + 8g + 4h + r puts the 8 keys of one operand in 16 contiguous bytes,
// so a lane fetches its V^T operand with one 16-byte read. Pairs (2i, 2i+1) stay adjacent.
__device__ __forceinline__ int vt_pos(int k) {
    return (k & ~31) | (((k >> 2) & 3) << 3) | (((k >> 4) & 1) << 2) | (k & 3);
}

// Row-major V tile (d_head 64, 128-byte rows): physical 8-byte unit = logical unit ^ vswz(row).
// The transposed reads of one 16-lane group touch rows 4a + {0..3} and four consecutive units,
// and the rows of a pair share a mask: with the mask moving a whole 4-unit block per row pair,
// the 32 lanes of two groups cover all 64 banks once.
__device__ __forceinline__ int vswz_m(int row) { return (row >> 1) & 3; }  // in 4-unit blocks
__device__ __forceinline__ int vswz(int row) { return vswz_m(row) << 2; }   // in 8-byte units
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) const uint16_t lds_cu16;

// Maximum over the lanes l, l^16, l^32, l^48 (the four lanes that hold one query's scores).
__device__ __forceinline__ float quad_max(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));  // {v of lane l & ~16, v of lane l | 16}
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));  // {l & 31, l | 32}
}

// Four waves per SIMD (at most 128 VGPRs): with 32 KB of LDS per work-group, four work-groups
// share a CU and cover one another's tile loads and barriers.
template <int DH, bool CLS>
__global__ __launch_bounds__(kWaves* kWave) __attribute__((amdgpu_waves_per_eu(4))) void attention_kernel(
    const uint16_t* __restrict__ qkv, const int32_t* __restrict__ seq_start, const int32_t* __restrict__ seq_len,
    const int32_t* __restrict__ work, int H, uint16_t* __restrict__ out, float scale_log2, int total) {
// The body is device code only: the host pass has no buffer-resource type, and a kernel whose
// body it cannot form would lose its host-side launch stub.
#if defined(__HIP_DEVICE_COMPILE__)
    constexpr int CPR = DH / 8;   // 16-byte chunks per head row
    constexpr int KS = DH / 32;   // MFMA k-steps over d_head
    constexpr int DT = DH / 16;   // 16-wide d blocks of the output
    // Two buffers, one array each: the compiler tracks direct-to-LDS loads per LDS variable, so
    // the loads into one buffer do not make it wait before reading the other.
    __shared__ __attribute__((aligned(16))) uint16_t sK0[kBKV * DH], sK1[kBKV * DH];
    // d_head 64: V tiles row-major (8-byte units XOR-swizzled by row pair, see vswz), read back
    // transposed by ds_read_b64_tr_b16; d_head 32: V^T rows staged through registers (vt_pos).
    constexpr bool VDIRECT = DH == 64;
    constexpr int VBUF = VDIRECT ? kBKV * DH : DH * kVtStride;
    __shared__ __attribute__((aligned(16))) uint16_t sV0[VBUF], sV1[VBUF];

    // Work-group w runs head w % H of work item w / H: the heads of one query tile are
    // adjacent, and the items come longest sequence first (the work list's order; slots
    // past the list's end hold length 0). CLS: item s is sequence s, one work-group per
    // (sequence, head) computing the first 32 queries (wave 0, exactly as in the full launch,
    // so the CLS query sees the same arithmetic) and writing the CLS row alone, to row s of a
    // one-row-per-sequence output.
    const int item = blockIdx.x / H, h = blockIdx.x - item * H;
    int s, seq0, L, q0;
    if constexpr (CLS) {
        s = item;
        seq0 = seq_start[s];
        L = seq_len[s];
        q0 = 0;
    } else {
        const int4 e = *reinterpret_cast<const int4*>(work + 4 * static_cast<size_t>(item));
        seq0 = e.x;
        L = e.y;
        q0 = e.z;
        s = e.w;
        if ((L <= 0) | (q0 < 0)) return;  // uniform; q0 >= 0 always, tested so the entry is loaded whole here
    }
    const int q_end = CLS ? (L < kQPerWave ? L : kQPerWave) : L;  // queries computed

    const int D = H * DH, D3 = 3 * D;
    const uint16_t* Qg = qkv + h * DH;
    const uint16_t* Kg = qkv + D + h * DH;
    const uint16_t* Vg = qkv + 2 * D + h * DH;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int g = lane >> 4, r16 = lane & 15;
    const int qw = q0 + wid * kQPerWave;
    const float lag = 8.0f / scale_log2;  // raw-score lag of the lazy running maximum

    // Query fragments (B operand of S^T = K Q^T): lane holds Q[query][8 d's of its k-group].
    bf16x8 qf[2][KS];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        int qi = qw + j * 16 + r16;
        qi = qi < L ? qi : L - 1;
        const uint16_t* row = Qg + static_cast<size_t>(seq0 + qi) * D3;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) qf[j][ks] = *reinterpret_cast<const bf16x8*>(row + ks * 32 + 8 * g);
    }

    f32x4 o[DT][2];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int j = 0; j < 2; ++j) o[dt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 lsum[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};  // row sums (every register)
    float m_run[2] = {-INFINITY, -INFINITY};
    bf16x8 ones;
#pragma unroll
    for (int e = 0; e < 8; ++e) ones[e] = static_cast<__bf16>(1.0f);

    // Staging of one 64-key tile. K goes from global memory straight into its LDS buffer
    // (direct-to-LDS loads, no registers): a wave-wide 16-byte load fills 64 / CPR consecutive
    // K rows, lane i writing the 16 bytes at offset 16 i, so lane i fetches the logical chunk
    // that the row swizzle places there; wave w fills rows [16 w, 16 w + 16). With d_head 64, V
    // takes the same route into a row-major tile; with d_head 32 it goes through registers as
    // pairs of rows (2 keys x 8 d) and is transposed into V^T on the way to LDS.
    // A tile wholly inside the sequence is addressed through a buffer resource over the packed
    // qkv rows (per-thread offsets of the first tile's rows plus the tile start as a scalar
    // offset, no per-tile address arithmetic); the sequence's last tile clamps its rows to the
    // last token, so no key or value of another sequence is ever read.
    constexpr int VCH = (kBKV / 2) * CPR;           // V units per tile
    constexpr int VPT = (VCH + kWaves * kWave - 1) / (kWaves * kWave);
    constexpr int KRL = kWave / CPR;                // K rows per direct load
    constexpr int KLW = 16 / KRL;                   // direct loads per wave per tile
    static_assert(KLW * KRL * kWaves == kBKV, "each wave fills 16 K rows");
    u32x4 rv0[VPT], rv1[VPT];
    const int wsc = __builtin_amdgcn_readfirstlane(wid);
    const bool offs32 = static_cast<size_t>(total) * D3 * 2 < (1ull << 31);
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(qkv), 0, offs32 ? total * D3 * 2 : 0, 0x00020000);
    int krow[KLW], kch[KLW], vch[KLW];
    uint32_t okb[KLW], ovd[KLW], ovb[VPT];
#pragma unroll
    for (int i = 0; i < KLW; ++i) {
        krow[i] = wsc * 16 + i * KRL + lane / CPR;
        kch[i] = (lane % CPR) ^ kswz<DH>(krow[i]);
        okb[i] = static_cast<uint32_t>(((seq0 + krow[i]) * D3 + D + h * DH + kch[i] * 8) * 2);
        vch[i] = (lane % CPR) ^ (vswz(krow[i]) >> 1);  // 16-byte chunk: the 8-byte swizzle in pairs
        ovd[i] = static_cast<uint32_t>(((seq0 + krow[i]) * D3 + 2 * D + h * DH + vch[i] * 8) * 2);
    }
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int u = tid + i * kWaves * kWave;
        ovb[i] = static_cast<uint32_t>(((seq0 + 2 * (u % (kBKV / 2))) * D3 + 2 * D + h * DH + (u / (kBKV / 2)) * 8) * 2);
    }
    typedef __attribute__((address_space(3))) void lds_t;
    auto gload = [&](int kv0, uint16_t* kd, uint16_t* vd) {
        uint16_t* k_s = kd + wsc * 16 * DH;
        if (offs32 && kv0 + kBKV <= L) {
            const int so = kv0 * D3 * 2;
#pragma unroll
            for (int i = 0; i < KLW; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_t*)(k_s + i * KRL * DH), 16, okb[i], so, 0, 0);
            if constexpr (VDIRECT) {
                uint16_t* v_d = vd + wsc * 16 * DH;
#pragma unroll
                for (int i = 0; i < KLW; ++i)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_t*)(v_d + i * KRL * DH), 16, ovd[i], so, 0, 0);
                return;
            }
#pragma unroll
            for (int i = 0; i < VPT; ++i) {
                if (VCH % (kWaves * kWave) == 0 || tid + i * kWaves * kWave < VCH) {
                    rv0[i] = __builtin_amdgcn_raw_buffer_load_b128(rq, ovb[i], so, 0);
                    rv1[i] = __builtin_amdgcn_raw_buffer_load_b128(rq, ovb[i] + D3 * 2, so, 0);
                }
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < KLW; ++i) {
            int tok = kv0 + krow[i];
            tok = tok < L ? tok : L - 1;
            __builtin_amdgcn_global_load_lds(Kg + static_cast<size_t>(seq0 + tok) * D3 + kch[i] * 8,
                                             (lds_t*)(k_s + i * KRL * DH), 16, 0, 0);
        }
        if constexpr (VDIRECT) {
            uint16_t* v_d = vd + wsc * 16 * DH;
#pragma unroll
            for (int i = 0; i < KLW; ++i) {
                int tok = kv0 + krow[i];
                tok = tok < L ? tok : L - 1;
                __builtin_amdgcn_global_load_lds(Vg + static_cast<size_t>(seq0 + tok) * D3 + vch[i] * 8,
                                                 (lds_t*)(v_d + i * KRL * DH), 16, 0, 0);
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
            const int u = tid + i * kWaves * kWave;
            if (VCH % (kWaves * kWave) == 0 || u < VCH) {
                const int tp = u % (kBKV / 2), ch = u / (kBKV / 2);
                int t0 = kv0 + 2 * tp, t1 = t0 + 1;
                t0 = t0 < L ? t0 : L - 1;
                t1 = t1 < L ? t1 : L - 1;
                rv0[i] = *reinterpret_cast<const u32x4*>(Vg + static_cast<size_t>(seq0 + t0) * D3 + ch * 8);
                rv1[i] = *reinterpret_cast<const u32x4*>(Vg + static_cast<size_t>(seq0 + t1) * D3 + ch * 8);
            }
        }
    };
    auto sstore = [&](uint16_t* v_s) {
        if constexpr (VDIRECT) return;
#pragma unroll
        for (int i = 0; i < VPT; ++i) {
            const int u = tid + i * kWaves * kWave;
            if (VCH % (kWaves * kWave) == 0 || u < VCH) {
                const int tp = u % (kBKV / 2), ch = u / (kBKV / 2);
                const u32x4 a = rv0[i], bb = rv1[i];
                const int pos = vt_pos(2 * tp);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    // (key 2tp, key 2tp+1) pairs for d = 8ch+2e and 8ch+2e+1
                    const uint32_t lo = __builtin_amdgcn_perm(bb[e], a[e], 0x05040100u);
                    const uint32_t hi = __builtin_amdgcn_perm(bb[e], a[e], 0x07060302u);
                    *reinterpret_cast<uint32_t*>(&v_s[(ch * 8 + 2 * e) * kVtStride + pos]) = lo;
                    *reinterpret_cast<uint32_t*>(&v_s[(ch * 8 + 2 * e + 1) * kVtStride + pos]) = hi;
                }
            }
        }
    };

    const int ntiles = (L + kBKV - 1) / kBKV;
    // Transposed V reads (d_head 64): lane 4r + q of a 16-lane group, d block dt, addresses key
    // row 4 g + r (+ 32 kc, + 16) at d columns 16 dt + 4 q, swizzled as the direct loads placed
    // it. The lane part is formed once, so each read's address is a short chain from its array.
    int vo[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        const int j16 = lane & 15, row = 4 * g + (j16 >> 2);
        vo[dt] = row * DH + (4 * (dt ^ vswz_m(row)) + (j16 & 3)) * 4;
    }
    gload(0, sK0, sV0);
    // Tile t: K and V in buffer t % 2 (k_s, vb), tile t + 1 loaded into the other (kn, vn);
    // unrolled twice so each buffer is a fixed array.
    auto tile = [&](int t, const uint16_t* k_s, uint16_t* vb, uint16_t* kn, uint16_t* vn) {
        const int kv0 = t * kBKV;
        // V of tile t into buffer t % 2 (last read in tile t-2, ordered by the barrier of tile t-1);
        // K of tile t was loaded into it directly. This wave's loads are all complete here, and
        // the barrier makes every wave's part of the tile visible.
        sstore(vb);
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), expcnt and lgkmcnt unconstrained: this wave's direct loads have landed
        __syncthreads();
        // The other buffer (tile t-1) is free: every wave has passed this barrier, so none still reads it.
        if (t + 1 < ntiles) gload(kv0 + kBKV, kn, vn);  // in flight while this tile is multiplied
        const uint16_t* v_s = vb;

        if (qw >= q_end) return;  // this wave's queries are all past the end (uniform per wave)

        // S^T = K Q^T: 4 key blocks x 2 query blocks (raw scores, unscaled).
        f32x4 sc[4][2];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
            const int row = tt * 16 + r16;
            bf16x8 kf[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int ch = ks * 4 + g;
                kf[ks] = *reinterpret_cast<const bf16x8*>(&k_s[row * DH + ((ch ^ kswz<DH>(row)) * 8)]);
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ks], qf[j][ks], acc, 0, 0, 0);
                sc[tt][j] = acc;
            }
        }
        if (kv0 + kBKV > L) {  // last tile only: keys past the end get -inf (uniform branch)
            const int valid = L - kv0;
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (tt * 16 + 4 * g + r >= valid) {
                        sc[tt][0][r] = -INFINITY;
                        sc[tt][1][r] = -INFINITY;
                    }
        }

        // Online softmax. The running maximum is kept in raw-score units; the scale
        // log2(e)/sqrt(d_head) enters once per score through the FMA inside exp2.
        // Lazy rescaling: the reference point m_run of a 16-query block only moves when one of
        // its queries meets a score more than lag = 8 / scale_log2 above it; then every query
        // of the block moves to its own running maximum and the block's accumulators are
        // rescaled. In between, p = 2^((s - m_run) * scale_log2) <= 2^8, which bf16 and the
        // fp32 sums hold with the same relative precision, and nothing is rescaled: after the
        // first tile a block rarely rescales again (with an exact running maximum nearly every
        // tile raised some query's maximum).
        bf16x8 pf[2][2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            float mx = fmaxf(fmaxf(sc[0][j][0], sc[0][j][1]), fmaxf(sc[0][j][2], sc[0][j][3]));
#pragma unroll
            for (int tt = 1; tt < 4; ++tt)
                mx = fmaxf(mx, fmaxf(fmaxf(sc[tt][j][0], sc[tt][j][1]), fmaxf(sc[tt][j][2], sc[tt][j][3])));
            mx = quad_max(mx);
            // m_run = -inf on the first tile: every query grows (each tile holds a valid key).
            if (__builtin_amdgcn_ballot_w64(mx > m_run[j] + lag) != 0) {
                const float m_new = fmaxf(m_run[j], mx);
                const float alpha = __builtin_amdgcn_exp2f((m_run[j] - m_new) * scale_log2);
                m_run[j] = m_new;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) o[dt][j] *= alpha;
                lsum[j] *= alpha;
            }
            const float nb = -m_run[j] * scale_log2;
            float p[4][4];
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r) p[tt][r] = __builtin_amdgcn_exp2f(fmaf(sc[tt][j][r], scale_log2, nb));
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                u32x4 w;
                w[0] = pack_bf16x2(p[2 * kc][0], p[2 * kc][1]);
                w[1] = pack_bf16x2(p[2 * kc][2], p[2 * kc][3]);
                w[2] = pack_bf16x2(p[2 * kc + 1][0], p[2 * kc + 1][1]);
                w[3] = pack_bf16x2(p[2 * kc + 1][2], p[2 * kc + 1][3]);
                pf[kc][j] = __builtin_bit_cast(bf16x8, w);
            }
        }

        // O^T += V^T P^T.
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = dt * 16 + r16;
#pragma unroll
            for (int kc = 0; kc < 2; ++kc) {
                // keys {kc*32 + 4g .. +3, kc*32 + 16 + 4g .. +3}: 16 contiguous bytes in V^T
                bf16x8 vf;
                if constexpr (VDIRECT) {
                    // Lane 4r + q of a 16-lane group points at key 32 kc + 4 g + r (then + 16),
                    // d-columns dt * 16 + 4 q .. +3; the transposed read hands lane i of the group
                    // those 4 keys of column dt * 16 + i: the 8 keys of the P^T operand's k-slots.
                    const lds_cu16* p0 = (lds_cu16*)(v_s) + vo[dt] + kc * 32 * DH;
                    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0));
                    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 16 * DH));
                    vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                } else {
                    vf = *reinterpret_cast<const bf16x8*>(&v_s[d * kVtStride + kc * 32 + 8 * g]);
                }
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    o[dt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[kc][j], o[dt][j], 0, 0, 0);
            }
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
            for (int j = 0; j < 2; ++j) lsum[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[kc][j], lsum[j], 0, 0, 0);
    };
    for (int t = 0; t < ntiles; t += 2) {
        tile(t, sK0, sV0, sK1, sV1);
        if (t + 1 < ntiles) tile(t + 1, sK1, sV1, sK0, sV0);
    }

    // Normalise and store: lane holds O[query j*16 + r16][d = dt*16 + 4g .. +3].
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const float inv = 1.0f / lsum[j][0];
        const int qi = qw + j * 16 + r16;
        if (CLS ? qi != 0 : qi >= L) continue;
        uint16_t* orow = out + static_cast<size_t>(CLS ? s : seq0 + qi) * D + h * DH;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            u32x2 pk;
            pk[0] = pack_bf16x2(o[dt][j][0] * inv, o[dt][j][1] * inv);
            pk[1] = pack_bf16x2(o[dt][j][2] * inv, o[dt][j][3] * inv);
            *reinterpret_cast<u32x2*>(orow + dt * 16 + 4 * g) = pk;
        }
    }
#endif
}

}  // namespace

hipError_t launch_attention(const uint16_t* qkv, SeqTable tab, int n, int total, int heads, int dh, uint16_t* out,
                            hipStream_t st, bool cls_only) {
    // The work list's capacity (an upper bound of sum_s ceil(len_s / kBQ)); surplus
    // work-groups find length 0 and exit at once.
    if (!cls_only && !tab.work) return hipErrorInvalidValue;
    const int items = cls_only ? n : attn_work_capacity(n, total);
    if (static_cast<long long>(items) * heads > 0x7fffffffLL) return hipErrorInvalidValue;
    const dim3 grid(items * heads), block(kWaves * kWave);
    const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(dh));
    auto go = [&](auto kernel) {
        return launch_kernel(kernel, grid, block, 0, st, qkv, tab.start, tab.len, tab.work, heads, out, scale_log2,
                             total);
    };
    if (dh == 64)
        ELIS_TRY(cls_only ? go(attention_kernel<64, true>) : go(attention_kernel<64, false>));
    else if (dh == 32)
        ELIS_TRY(cls_only ? go(attention_kernel<32, true>) : go(attention_kernel<32, false>));
    else
        return hipErrorInvalidValue;
    return hipSuccess;
}

}  // namespace elis
