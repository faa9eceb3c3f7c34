// Dense layers of the encoder on the CDNA4 matrix cores:
//   out[m, n] = epilogue( sum_k x[m, k] * w[n, k] + bias[n] )
// x is the activation, bf16 [M, K] row-major; w is the weight, bf16 [N, K]
// row-major ([out, in]); both operands are K-contiguous. fp32 accumulation.
// Epilogues: bf16 out; bf16 out after GELU; fp32 out plus a residual, which is
// either an fp32 matrix or a LayerNorm output rebuilt from its pre-norm rows and
// row statistics (Residual in kernels.h).
//
// Two kernel families; launch_gemm plans each product (plan_gemm: one launch, or a
// launch of large tiles over whole rounds plus one of small tiles over the remaining rows):
//   gemm_kernel        register-staged k-slabs, 16 x 16 x 32 MFMA blocks; for N that
//                      is an odd multiple of 64;
//   gemm_sched_kernel  k-slabs go HBM -> LDS with global_load_lds_dwordx4 (no register
//                      staging), 32 x 32 x 16 MFMA blocks, a hand-scheduled k-loop
//                      (operand fragments double-buffered in registers, MFMAs of the
//                      last k-step of a slab issued after the slab barrier) and an
//                      epilogue staged through LDS for full-line stores; tiles of
//                      256 x 256, 128 x 128, 64 x 128 and 64 x 64.
//
// LDS layout. A k-slab row of 64 bf16 is eight 16-byte chunks; the chunk index
// is XOR-swizzled with the row so the rows one MFMA operand read touches fall on
// different banks (see swz).
//
// Operand order. The MFMA is issued as (weight fragment, activation
// fragment), which computes the transposed tile: lane l then holds 4
// consecutive output columns of one output row, so the epilogue reads
// bias / residual and writes the output as 16-byte (fp32) or 8-byte (bf16)
// vectors.
//
// Work-group order. The hardware hands consecutive work-group ids round-robin
// to the 8 XCDs (each with its own L2). Ids are remapped so every XCD gets one
// contiguous range of tiles, grouped GROUP_M tile rows at a time: the tiles an
// XCD runs together share activation rows and weight columns in its L2.
#include <atomic>
#include <type_traits>

#include "gemm_common.h"
#include "kernels.h"

namespace elis {

namespace {

using namespace gemm;

constexpr int kBK = 64;

template <int EPI>
constexpr bool kF32Out = EPI == ELIS_EPI_BIAS_RES_F32 || EPI == kEpiResLn || EPI == kEpiResLnFfn2;
template <int EPI>
constexpr bool kResLn = EPI == kEpiResLn || EPI == kEpiResLnFfn2;
constexpr bool kResLnCode(int epi) { return epi == kEpiResLn || epi == kEpiResLnFfn2; }

// Residual of 4 consecutive columns n..n+3 of row m, given the 4 values h of res.x there.
template <int EPI>
__device__ __forceinline__ f32x4 residual4(const Residual& res, f32x4 h, int m, int n) {
    if constexpr (kResLn<EPI>) {
        const float2 st = res.stats[m];
        const f32x4 g = *reinterpret_cast<const f32x4*>(res.g + n);
        const f32x4 b = *reinterpret_cast<const f32x4*>(res.b + n);
#pragma unroll
        for (int c = 0; c < 4; ++c) h[c] = fmaf((h[c] - st.x) * st.y, g[c], b[c]);
    }
    return h;
}


// LDS chunk swizzle of the direct-to-LDS kernels: physical 16-byte chunk = logical chunk ^ swz(row).
// Measured free of bank conflicts on gfx950 for both 16-row and 32-row fragment reads (the
// plain row & 7 form conflicts 4-way on 32-row reads).
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

// GELU(x) = x * Phi(x) = max(x, 0) - a * Phi(-a) with a = |x| (as Phi(-a) = 1 - Phi(a)), so no
// branch or select on the sign. log2 Phi(-a) is smooth on [0, 5]: a degree-7 polynomial fitted
// there by weighted least squares (weight a * Phi(-a), the error it makes in GELU) gives Phi(-a)
// through one exp2. Past a = 5 the clamp leaves less than 5 * Phi(-5) < 1.5e-6 of error. Over
// all floats the result is within 1.5e-6 absolute and 3e-5 relative (where |GELU| > 1e-3) of
// x * Phi(x), far below the bf16 rounding of the output: one exp2, eight FMAs, a min and a max
// (a rational erf approximation needs a reciprocal as well, and measured 5% slower on FFN1).
__device__ __forceinline__ float gelu_erf(float x) {
    constexpr float c0 = -9.999995232e-01f, c1 = -1.151127219e+00f, c2 = -4.590456784e-01f,
                    c3 = -5.294791982e-02f, c4 = 7.674183231e-03f, c5 = -5.793952732e-04f,
                    c6 = -1.149886975e-05f, c7 = 4.121166967e-06f;
    const float a = fminf(fabsf(x), 5.0f);
    const float q = fmaf(fmaf(fmaf(fmaf(fmaf(fmaf(fmaf(c7, a, c6), a, c5), a, c4), a, c3), a, c2), a, c1), a, c0);
    return fmaf(-a, __builtin_amdgcn_exp2f(q), fmaxf(x, 0.f));
}


template <int BM, int BN, int WM, int WN, int MI, int EPI>
__global__ __launch_bounds__(WM* WN* kWave) void gemm_kernel(const uint16_t* __restrict__ A,
                                                             const uint16_t* __restrict__ B,
                                                             const float* __restrict__ bias,
                                                             Residual res, void* __restrict__ out,
                                                             int M, int N, int K) {
    typedef Mfma<MI> MF;
    typedef typename MF::acc_t acc_t;
    constexpr int NT = WM * WN * kWave;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / MI, FN = TN / MI;
    constexpr int KSTEPS = kBK / MF::kDepth;
    constexpr int GROUPS = kWave / MI;  // lane groups along k (4 for MI 16, 2 for MI 32)
    constexpr int ACH = BM * 8 / NT, BCH = BN * 8 / NT;  // 16-byte chunks per thread per k-slab
    static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile must split evenly over the threads");
    static_assert(TM % MI == 0 && TN % MI == 0, "wave tile must be a multiple of the MFMA block");

    __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * kBK];
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * kBK];

    const int tiles_n = N / BN;
    const int tiles_m = (M + BM - 1) / BM;
    const int t = xcd_remap(blockIdx.x, tiles_m * tiles_n);
    const int m0 = (t / tiles_n) * BM, n0 = (t % tiles_n) * BN;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int wm = wid / WN, wn = wid % WN;

    // Per-thread global source pointers and LDS destinations of the k-slab chunks.
    const uint16_t* ga[ACH];
    const uint16_t* gb[BCH];
    int la[ACH], lb[BCH];
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
        const int id = tid + i * NT, row = id >> 3, c = id & 7;
        const int gr = (m0 + row < M) ? m0 + row : M - 1;  // ragged tail: re-read the last row
        ga[i] = A + static_cast<size_t>(gr) * K + c * 8;
        la[i] = row * kBK + ((c ^ (row & 7)) * 8);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
        const int id = tid + i * NT, row = id >> 3, c = id & 7;
        gb[i] = B + static_cast<size_t>(n0 + row) * K + c * 8;
        lb[i] = row * kBK + ((c ^ (row & 7)) * 8);
    }

    u32x4 ra[ACH], rb[BCH];
    acc_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < MF::kRegs; ++r) acc[i][j][r] = 0.f;

    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < ACH; ++i) ra[i] = *reinterpret_cast<const u32x4*>(ga[i] + k0);
#pragma unroll
        for (int i = 0; i < BCH; ++i) rb[i] = *reinterpret_cast<const u32x4*>(gb[i] + k0);
    };
    auto sstore = [&](int stg) {
#pragma unroll
        for (int i = 0; i < ACH; ++i) *reinterpret_cast<u32x4*>(&sA[stg][la[i]]) = ra[i];
#pragma unroll
        for (int i = 0; i < BCH; ++i) *reinterpret_cast<u32x4*>(&sB[stg][lb[i]]) = rb[i];
    };

    const int KT = K / kBK;
    gload(0);
    sstore(0);
    __syncthreads();

    const int rl = lane % MI, kg = lane / MI;
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT) gload((kt + 1) * kBK);
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            const int c = ks * GROUPS + kg;  // 16-byte chunk (8 k values) this lane feeds
            bf16x8 af[FM], bfr[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int row = wm * TM + i * MI + rl;
                af[i] = *reinterpret_cast<const bf16x8*>(&sA[cur][row * kBK + ((c ^ (row & 7)) * 8)]);
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int row = wn * TN + j * MI + rl;
                bfr[j] = *reinterpret_cast<const bf16x8*>(&sB[cur][row * kBK + ((c ^ (row & 7)) * 8)]);
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j) acc[i][j] = MF::run(bfr[j], af[i], acc[i][j]);
        }
        if (kt + 1 < KT) sstore(cur ^ 1);
        __syncthreads();
    }

    // Epilogue. Lane holds, for output row m = rl of block i, groups of 4 consecutive
    // columns: MI 16: one group at 4*kg; MI 32: four groups at 8*q + 4*kg.
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = m0 + wm * TM + i * MI + rl;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int q = 0; q < MF::kRegs / 4; ++q) {
                const int n = n0 + wn * TN + j * MI + 8 * q + 4 * kg;
                f32x4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * q + r];
                v += *reinterpret_cast<const f32x4*>(bias + n);
                const size_t o = static_cast<size_t>(m) * N + n;
                if constexpr (kF32Out<EPI>) {
                    v += residual4<EPI>(res, *reinterpret_cast<const f32x4*>(res.x + o), m, n);
                    *reinterpret_cast<f32x4*>(static_cast<float*>(out) + o) = v;
                } else {
                    if constexpr (EPI == ELIS_EPI_BIAS_GELU_BF16) {
#pragma unroll
                        for (int c = 0; c < 4; ++c) v[c] = gelu_erf(v[c]);
                    }
                    u32x2 p;
                    p[0] = pack_bf16x2(v[0], v[1]);
                    p[1] = pack_bf16x2(v[2], v[3]);
                    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + o) = p;
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Direct-to-LDS loading: k-slabs go from HBM straight into LDS (global_load_lds_dwordx4, no
// register staging), S stages deep, so S-1 slabs are in flight while one is multiplied.
// Each thread waits (vmcnt) only for its own loads of the slab about to be consumed; the
// barrier that follows makes every thread's part of that slab visible and also guarantees
// that every wave has finished reading the stage the next loads will overwrite.


// Tile index -> (tile row, tile col), grouping GM tile rows so that the tiles running
// together on one XCD share a small set of A rows and B columns (L2 reuse).
__device__ __forceinline__ void grouped_tile(int t, int tiles_m, int tiles_n, int gm, int& tm, int& tn) {
    const int per_group = gm * tiles_n;
    const int g = t / per_group, first = g * gm;
    const int rows = (tiles_m - first) < gm ? (tiles_m - first) : gm;
    const int r = t - g * per_group;
    tm = first + r % rows;
    tn = r / rows;
}

// ---------------------------------------------------------------------------------------------
// Scheduled variant: 4 waves (2 x 2), each owning a (BM/2) x (BN/2) block of MFMA tiles; two
// LDS stages filled by direct-to-LDS loads. A 64-deep k-slab is consumed in k-steps whose
// operand fragments are double-buffered in registers, so the LDS reads of the next k-step
// run under the MFMAs of the current one. The slab two steps ahead is requested right after
// the barrier that frees its stage (before the last k-step of the current slab), so a load
// has one full slab of MFMA work to arrive. sched_group_barrier spreads the LDS reads and the
// direct loads evenly between the MFMAs.
//
// LDS chunk swizzle: physical chunk = logical chunk ^ ((row >> 1) & 7). Measured free of bank
// conflicts on gfx950 for both the 16-row (16x16x32) and 32-row (32x32x16) fragment reads;
// the plain (row & 7) form conflicts 4-way on the 32-row reads.


template <int BM, int BN, int WM, int WN, int MI, int EPI, int OCC = 1, int S = 2>
__global__ __launch_bounds__(WM* WN* kWave) __attribute__((amdgpu_waves_per_eu(OCC * WM * WN / 4, OCC * WM * WN / 4))) void gemm_sched_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ B, const float* __restrict__ bias,
    Residual res, void* __restrict__ out, int M, int N, int K, int group_m) {
    typedef Mfma<MI> MF;
    typedef typename MF::acc_t acc_t;
    constexpr int BK = kBK;              // k-slab depth: 64 (eight 16-byte chunks per row)
    constexpr int NW = WM * WN;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / MI, FN = TN / MI;
    constexpr int KS = BK / MF::kDepth;    // k-steps per slab
    constexpr int GROUPS = kWave / MI;     // lane groups along k
    constexpr int CPR = BK / 8;            // 16-byte chunks per slab row
    constexpr int RPI = kWave / CPR;       // slab rows covered by one wave-wide 16-byte load
    constexpr int LA = BM / RPI / NW, LB = BN / RPI / NW;  // direct loads per wave per stage
    static_assert(BM % (RPI * NW) == 0 && BN % (RPI * NW) == 0, "rows must split over the waves");
    constexpr int STAGE = (BM + BN) * BK;
    constexpr int NMF = FM * FN, NRD = FM + FN, NGL = LA + LB;
    static_assert(KS % 2 == 0, "fragment buffers alternate per k-step");
    static_assert(S >= 2 && S * NGL < 64, "pipeline depth");
    __shared__ __attribute__((aligned(1024))) uint16_t smem[S * STAGE];

    const int tiles_n = N / BN;
    const int tiles_m = (M + BM - 1) / BM;
    int tm, tn;
    grouped_tile(xcd_remap(blockIdx.x, tiles_m * tiles_n), tiles_m, tiles_n, group_m, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wm = wid / WN, wn = wid % WN;
    auto sw = [](int row) { return (row >> 1) & (CPR - 1); };

    const uint16_t* ga[LA];
    const uint16_t* gb[LB];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int row = (wid * LA + i) * RPI + lane / CPR;
        const int c = (lane % CPR) ^ sw(row);
        const int gr = (m0 + row < M) ? m0 + row : M - 1;
        ga[i] = A + static_cast<size_t>(gr) * K + c * 8;
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int row = (wid * LB + i) * RPI + lane / CPR;
        const int c = (lane % CPR) ^ sw(row);
        gb[i] = B + static_cast<size_t>(n0 + row) * K + c * 8;
    }
    auto issue = [&](int kt) {
        uint16_t* st = smem + (kt % S) * STAGE;
        const int k0 = kt * BK;
#pragma unroll
        for (int i = 0; i < LA; ++i) load_lds_16(ga[i] + k0, st + (wid * LA + i) * RPI * BK);
#pragma unroll
        for (int i = 0; i < LB; ++i) load_lds_16(gb[i] + k0, st + BM * BK + (wid * LB + i) * RPI * BK);
    };

    const int rl = lane % MI, kg = lane / MI;
    int offa[FM], offb[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) offa[i] = (wm * TM + i * MI + rl) * BK;
#pragma unroll
    for (int j = 0; j < FN; ++j) offb[j] = BM * BK + (wn * TN + j * MI + rl) * BK;
    const int rs = sw(rl);  // fragment rows start at multiples of 16, so sw(row) == sw(rl)

    bf16x8 fa[2][FM], fb[2][FN];
    auto load_frags = [&](int buf, int stage, int ks) {
        const uint16_t* st = smem + stage * STAGE;
        const int c = ((ks * GROUPS + kg) ^ rs) * 8;
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[buf][i] = *reinterpret_cast<const bf16x8*>(st + offa[i] + c);
#pragma unroll
        for (int j = 0; j < FN; ++j) fb[buf][j] = *reinterpret_cast<const bf16x8*>(st + offb[j] + c);
    };

    acc_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < MF::kRegs; ++r) acc[i][j][r] = 0.f;

    auto mfma_all = [&](int buf) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j) acc[i][j] = MF::run(fb[buf][j], fa[buf][i], acc[i][j]);
    };

    const int KT = K / BK;
    // Prologue: every stage gets a slab (slabs 0 .. S-1); wait for slab 0 only.
#pragma unroll
    for (int p = 0; p < S; ++p)
        if (p < KT) issue(p);
    if (KT >= S) wait_vmcnt<(S - 1) * NGL>();
    else wait_vmcnt<0>();
    block_sync_lds();
    load_frags(0, 0, 0);

    // One slab. WAIT: slabs still allowed in flight once slab kt+1 has landed; ISSUE: request
    // slab kt+S into the stage slab kt frees; NEXT: slab kt+1 exists (read its first
    // fragments). All compile-time, so the steady-state loop is straight-line code.
    auto slab = [&](int kt, auto wait_c, auto issue_c, auto next_c) {
        constexpr int WAIT = decltype(wait_c)::value;
        constexpr bool ISSUE = decltype(issue_c)::value, NEXT = decltype(next_c)::value;
        const int cur = kt % S;
#pragma unroll
        for (int ks = 0; ks < KS - 1; ++ks) {
            load_frags((ks + 1) & 1, cur, ks + 1);
            mfma_all(ks & 1);
            interleave_step<0, NMF, 0, NRD, 0>();
        }
        // Slab kt+1 has landed and every wave's reads of stage `cur` are complete.
        wait_vmcnt<WAIT * NGL>();
        wait_lgkm<0>();
        block_sync_lds();
        if constexpr (ISSUE) issue(kt + S);
        if constexpr (NEXT) load_frags(0, (kt + 1) % S, 0);
        mfma_all((KS - 1) & 1);
        interleave_step<0, NMF, ISSUE ? NGL : 0, NEXT ? NRD : 0, 1>();
    };
    typedef std::integral_constant<bool, true> T_;
    typedef std::integral_constant<bool, false> F_;
    typedef std::integral_constant<int, S - 2> WS_;
    typedef std::integral_constant<int, 0> W0_;
    int kt = 0;
    for (; kt + S < KT; ++kt) slab(kt, WS_(), T_(), T_());
    for (; kt + 1 < KT; ++kt) slab(kt, W0_(), F_(), T_());
    slab(kt, W0_(), F_(), F_());

    // Epilogue through LDS: each wave stages one 32-row block row of its output tile (bias,
    // activation / residual applied), then writes it back as whole rows, 16 bytes per lane,
    // so every store instruction covers full cache lines. bf16 outputs are stored
    // non-temporally: they stream past the caches that hold the next tiles' operands (1% per
    // predictor pass, up to 9% for a single GEMM). fp32 outputs (the pre-LayerNorm rows) are
    // stored normally: the LayerNorm that reads them next then finds part of them in the
    // memory-side cache (LayerNorm 21.4 -> 20.0 us at 24K tokens, 0.8% per pass).
    static_assert(MI == 32, "staged epilogue assumes 32-row MFMA blocks");
    constexpr bool F32OUT = kF32Out<EPI>;
    constexpr int EB = F32OUT ? 4 : 2;          // output element bytes
    constexpr int ROWB = TN * EB;               // bytes of one wave-tile row
    constexpr int PITCH = ROWB + 16;            // padded LDS row pitch
    constexpr int LPR = ROWB / 16;              // lanes per row on read-back
    constexpr int RPR = kWave / LPR;            // rows per read-back instruction
    static_assert(NW * 32 * PITCH <= S * STAGE * 2, "staging must fit in the stage buffers");
    block_sync_lds();  // every wave is done with the stage buffers
    char* stg = reinterpret_cast<char*>(smem) + wid * 32 * PITCH;
    // On read-back a lane always covers the same 16 output bytes of a row: columns nl ...
    const int ch = lane % LPR;
    const int nl = n0 + wn * TN + ch * (16 / EB);
    f32x4 gl, bl;  // LayerNorm g, b of those columns (LayerNorm-form residual)
    if constexpr (kResLn<EPI>) {
        gl = *reinterpret_cast<const f32x4*>(res.g + nl);
        bl = *reinterpret_cast<const f32x4*>(res.b + nl);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = j * MI + 8 * q + 4 * kg;
                f32x4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * q + r];
                v += *reinterpret_cast<const f32x4*>(bias + n0 + wn * TN + col);
                if constexpr (F32OUT) {
                    *reinterpret_cast<f32x4*>(stg + rl * PITCH + col * 4) = v;
                } else {
                    if constexpr (EPI == ELIS_EPI_BIAS_GELU_BF16) {
#pragma unroll
                        for (int c = 0; c < 4; ++c) v[c] = gelu_erf(v[c]);
                    }
                    u32x2 pk;
                    pk[0] = pack_bf16x2(v[0], v[1]);
                    pk[1] = pack_bf16x2(v[2], v[3]);
                    *reinterpret_cast<u32x2*>(stg + rl * PITCH + col * 2) = pk;
                }
            }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_wave_barrier();
        asm volatile("" ::: "memory");
        constexpr int NRR = 32 / RPR;  // read-back rows per lane per block row
        if constexpr (F32OUT) {
            // All residual vectors (and row statistics) of the block row are requested first.
            f32x4 hv[NRR];
            float2 sv[NRR];
#pragma unroll
            for (int rr = 0; rr < NRR; ++rr) {
                const int m = m0 + wm * TM + i * MI + rr * RPR + lane / LPR;
                const int mc = m < M ? m : M - 1;  // rows past the end load a valid row, store nothing
                hv[rr] = *reinterpret_cast<const f32x4*>(res.x + static_cast<size_t>(mc) * N + nl);
                if constexpr (kResLn<EPI>) sv[rr] = res.stats[mc];
            }
#pragma unroll
            for (int rr = 0; rr < NRR; ++rr) {
                const int row = rr * RPR + lane / LPR;
                const int m = m0 + wm * TM + i * MI + row;
                const u32x4 d = *reinterpret_cast<const u32x4*>(stg + row * PITCH + ch * 16);
                if (m < M) {
                    f32x4 h = hv[rr];
                    if constexpr (kResLn<EPI>) {
#pragma unroll
                        for (int c = 0; c < 4; ++c) h[c] = fmaf((h[c] - sv[rr].x) * sv[rr].y, gl[c], bl[c]);
                    }
                    const f32x4 v = __builtin_bit_cast(f32x4, d) + h;
                    *reinterpret_cast<f32x4*>(static_cast<float*>(out) + static_cast<size_t>(m) * N + nl) = v;
                }
            }
        } else {
#pragma unroll
            for (int rr = 0; rr < NRR; ++rr) {
                const int row = rr * RPR + lane / LPR;
                const int m = m0 + wm * TM + i * MI + row;
                const u32x4 d = *reinterpret_cast<const u32x4*>(stg + row * PITCH + ch * 16);
                if (m < M) __builtin_nontemporal_store(d, reinterpret_cast<u32x4*>(static_cast<uint16_t*>(out) + static_cast<size_t>(m) * N + nl));
            }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_wave_barrier();
        asm volatile("" ::: "memory");
    }
}

template <int BM, int BN, int WM, int WN, int MI, int OCC = 1, int S = 2>
hipError_t launch_sched(const uint16_t* x, const uint16_t* w, const float* bias, Residual res, int m, int n,
                        int k, int epi, void* out, hipStream_t st, int group_m) {
    const dim3 grid(((m + BM - 1) / BM) * (n / BN)), block(WM * WN * kWave);
    switch (epi) {
        case ELIS_EPI_BIAS_BF16:
            ELIS_TRY(launch_kernel((gemm_sched_kernel<BM, BN, WM, WN, MI, ELIS_EPI_BIAS_BF16, OCC, S>), grid, block, 0, st, x, w, bias,
                               res, out, m, n, k, group_m));
            break;
        case ELIS_EPI_BIAS_GELU_BF16:
            ELIS_TRY(launch_kernel((gemm_sched_kernel<BM, BN, WM, WN, MI, ELIS_EPI_BIAS_GELU_BF16, OCC, S>), grid, block, 0, st, x, w,
                               bias, res, out, m, n, k, group_m));
            break;
        case ELIS_EPI_BIAS_RES_F32:
            ELIS_TRY(launch_kernel((gemm_sched_kernel<BM, BN, WM, WN, MI, ELIS_EPI_BIAS_RES_F32, OCC, S>), grid, block, 0, st, x, w,
                               bias, res, out, m, n, k, group_m));
            break;
        case kEpiResLn:
            ELIS_TRY(launch_kernel((gemm_sched_kernel<BM, BN, WM, WN, MI, kEpiResLn, OCC, S>), grid, block, 0, st, x, w, bias, res,
                               out, m, n, k, group_m));
            break;
        case kEpiResLnFfn2:
            ELIS_TRY(launch_kernel((gemm_sched_kernel<BM, BN, WM, WN, MI, kEpiResLnFfn2, OCC, S>), grid, block, 0, st, x, w, bias, res,
                               out, m, n, k, group_m));
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipSuccess;
}

template <int BM, int BN, int WM, int WN, int MI>
hipError_t launch_tile(const uint16_t* x, const uint16_t* w, const float* bias, Residual res, int m, int n,
                       int k, int epi, void* out, hipStream_t st) {
    const dim3 grid(((m + BM - 1) / BM) * (n / BN)), block(WM * WN * kWave);
    switch (epi) {
        case ELIS_EPI_BIAS_BF16:
            ELIS_TRY(launch_kernel((gemm_kernel<BM, BN, WM, WN, MI, ELIS_EPI_BIAS_BF16>), grid, block, 0, st, x, w,
                               bias, res, out, m, n, k));
            break;
        case ELIS_EPI_BIAS_GELU_BF16:
            ELIS_TRY(launch_kernel((gemm_kernel<BM, BN, WM, WN, MI, ELIS_EPI_BIAS_GELU_BF16>), grid, block, 0, st, x,
                               w, bias, res, out, m, n, k));
            break;
        case ELIS_EPI_BIAS_RES_F32:
            ELIS_TRY(launch_kernel((gemm_kernel<BM, BN, WM, WN, MI, ELIS_EPI_BIAS_RES_F32>), grid, block, 0, st, x, w,
                               bias, res, out, m, n, k));
            break;
        case kEpiResLn:
            ELIS_TRY(launch_kernel((gemm_kernel<BM, BN, WM, WN, MI, kEpiResLn>), grid, block, 0, st, x, w, bias,
                               res, out, m, n, k));
            break;
        case kEpiResLnFfn2:
            ELIS_TRY(launch_kernel((gemm_kernel<BM, BN, WM, WN, MI, kEpiResLnFfn2>), grid, block, 0, st, x, w, bias,
                               res, out, m, n, k));
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipSuccess;
}

}  // namespace

// Tile configurations (ids are internal; benchmarks sweep them).
hipError_t launch_gemm_config(int cfg, int group_m, const uint16_t* x, const uint16_t* w, const float* bias,
                              Residual res, int m, int n, int k, int epi, void* out, hipStream_t st) {
    switch (cfg) {
        case 1: return launch_tile<128, 64, 2, 2, 16>(x, w, bias, res, m, n, k, epi, out, st);
        case 21: return launch_sched<256, 256, 2, 4, 32>(x, w, bias, res, m, n, k, epi, out, st, group_m);
        case 32: return launch_sched<128, 128, 2, 2, 32, 2>(x, w, bias, res, m, n, k, epi, out, st, group_m);
        case 33: return launch_sched<64, 128, 2, 2, 32, 2>(x, w, bias, res, m, n, k, epi, out, st, group_m);
        case 34: return launch_sched<64, 128, 2, 2, 32, 1, 4>(x, w, bias, res, m, n, k, epi, out, st, group_m);
        case 35: return launch_sched<64, 64, 2, 2, 32, 4, 2>(x, w, bias, res, m, n, k, epi, out, st, group_m);
        case 36: return launch_sched<64, 64, 2, 2, 32, 2, 4>(x, w, bias, res, m, n, k, epi, out, st, group_m);
        default: return hipErrorInvalidValue;
    }
}

namespace {
struct TileShape {
    int cfg, bm, bn, wgs_per_cu;
};
constexpr TileShape kTileShapes[] = {{1, 128, 64, 2},   {21, 256, 256, 1}, {32, 128, 128, 2}, {33, 64, 128, 2},
                                     {34, 64, 128, 1},  {35, 64, 64, 4},   {36, 64, 64, 2}};
}  // namespace

void gemm_config_tile(int cfg, int* bm, int* bn, int* wgs_per_cu) {
    *bm = *bn = *wgs_per_cu = 0;
    for (const TileShape& t : kTileShapes)
        if (t.cfg == cfg) *bm = t.bm, *bn = t.bn, *wgs_per_cu = t.wgs_per_cu;
}

int gemm_config_of_tile(int bm, int bn, int wgs_per_cu) {
    for (const TileShape& t : kTileShapes)
        if (t.bm == bm && t.bn == bn && t.wgs_per_cu == wgs_per_cu) return t.cfg;
    return -1;
}

// Compute units of the current device (the launch-time model below needs it). A device property,
// looked up once per device; the cache is safe to read and fill from several host threads.
int device_cus() {
    static std::atomic<int> cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cus[dev].load(std::memory_order_relaxed);
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cus[dev].store(v, std::memory_order_relaxed);
    }
    return v;
}

namespace {

// Launch-time model of the scheduled configurations, in microseconds on MI355X (256 CUs),
// fitted to medians of repeated timings of the BERT-base and XLM-R-large encoder GEMMs
// (K = 768 .. 4096, one to four rounds of tiles; all six configurations timed on one box).
// A launch whose tiles fill R rounds of work-group slots (work-groups per CU x CUs), the last
// one a fraction f full, takes part(f) for R = 1, else t1 + (R - 2) * beta + part(f)
// - (t1 - beta) * f; part is piecewise linear through lat (a lone tile, f -> 0), th (f = 1/2)
// and t1 (f = 1), beta is the cost of one more full round. Each quantity is a + s * K / 64: the slope per 64-deep k-slab is shared by the
// epilogue kinds, the intercept is per kind (bf16, bf16 + GELU, fp32 + residual). The 64-row
// tiles are priced only up to the four rounds they were timed on and are not offered past
// that. Over every single and split plan of those shapes at 35 sizes (M = 1K .. 92K), timed
// one by one, the plans it picks take 0.25-0.4% more time in total than the fastest ones
// measured (two boxes).
struct TileModel {
    int cfg, bm, bn, occ, max_rounds;  // max_rounds: 0 = any; else the fitted range
    float s[4];     // lat, th, t1, beta: slope per k-slab
    float a[3][4];  // intercept per epilogue kind
};
constexpr TileModel kTileModels[] = {
    {21, 256, 256, 1, 0, {1.178f, 1.375f, 1.770f, 1.693f},
     {{6.05f, 5.97f, 5.72f, 4.21f}, {11.77f, 11.79f, 11.15f, 10.12f}, {10.41f, 14.62f, 20.49f, 26.70f}}},
    {32, 128, 128, 2, 0, {0.535f, 0.614f, 0.991f, 1.073f},
     {{3.63f, 3.63f, 4.11f, 2.01f}, {5.24f, 6.32f, 7.50f, 4.91f}, {4.94f, 9.43f, 12.78f, 12.17f}}},
    {33, 64, 128, 2, 4, {0.363f, 0.556f, 0.594f, 0.754f},
     {{2.94f, 2.37f, 3.95f, 0.42f}, {3.69f, 1.94f, 4.59f, 1.10f}, {3.45f, 3.46f, 8.15f, 3.02f}}},
    {34, 64, 128, 1, 4, {0.340f, 0.395f, 0.436f, 0.353f},
     {{3.49f, 2.78f, 2.74f, 2.45f}, {4.11f, 3.68f, 3.67f, 3.50f}, {4.17f, 3.89f, 5.00f, 4.40f}}},
    {35, 64, 64, 4, 4, {0.227f, 0.481f, 0.757f, 0.844f},
     {{2.78f, 1.95f, 3.73f, -0.05f}, {3.11f, 1.74f, 4.15f, 0.50f}, {3.24f, 3.77f, 6.41f, 1.22f}}},
    {36, 64, 64, 2, 4, {0.251f, 0.259f, 0.411f, 0.393f},
     {{2.47f, 2.85f, 3.10f, 1.40f}, {3.23f, 3.40f, 3.12f, 1.82f}, {2.97f, 4.12f, 4.86f, 2.60f}}},
};
constexpr float kSecondLaunchUs = 1.0f;  // dispatch cost of the remainder launch

double model_us(const TileModel& t, int kind, long long m, int n, int k, long long cus) {
    if (m <= 0) return 0.0;
    const long long tiles = (m + t.bm - 1) / t.bm * (n / t.bn), slots = t.occ * cus;
    const long long rounds = (tiles + slots - 1) / slots;
    // The small tiles were timed over one to four rounds only; past that their cost is not
    // extrapolated (their many-round behaviour differs) and they are not offered.
    if (t.max_rounds && rounds > t.max_rounds) return 1e30;
    const double f = static_cast<double>(tiles - (rounds - 1) * slots) / static_cast<double>(slots);
    double v[4];
    for (int q = 0; q < 4; ++q) v[q] = t.a[kind][q] + t.s[q] * (k / 64.0);
    const double part = f <= 0.5 ? v[0] + (v[1] - v[0]) * (f / 0.5) : v[1] + (v[2] - v[1]) * ((f - 0.5) / 0.5);
    if (rounds == 1) return part;
    // First round t1, full rounds after it beta each (they overlap the one before), and a last
    // round f full that overlaps the one before it by (t1 - beta) * f.
    return v[2] + static_cast<double>(rounds - 2) * v[3] + part - (v[2] - v[3]) * f;
}

}  // namespace

// The plan of one product: a single launch of one configuration, or (main, m1, rest): rows
// [0, m1) with `main` in whole rounds of tiles and rows [m1, m) with the smaller-tile `rest`,
// whichever the launch-time model above prices lowest. A 256 x 256 round costs about as much
// as two rounds of the 128 x 128 pairs, but a round that is only partly filled costs nearly a
// full one, so the rows past the last full round of large tiles go to a configuration whose
// tiles are small enough to finish them in one short round.
GemmPlan plan_gemm(int m, int n, int k, int epi) {
    const bool f32out = epi == ELIS_EPI_BIAS_RES_F32 || kResLnCode(epi);
    if (n % 128 != 0) return {1, m, 0};
    const int kind = f32out ? 2 : (epi == ELIS_EPI_BIAS_GELU_BF16 ? 1 : 0);
    const long long cus = device_cus();
    GemmPlan best{21, m, 0};
    double best_us = -1.0;
    for (const TileModel& main : kTileModels) {
        if (n % main.bn != 0) continue;
        const double t = model_us(main, kind, m, n, k, cus);
        if (best_us < 0.0 || t < best_us) {
            best_us = t;
            best = {main.cfg, m, 0};
        }
        // Whole rows of tiles that fill whole rounds.
        const long long per_row = n / main.bn, slots = main.occ * cus;
        const long long tiles = (static_cast<long long>(m) + main.bm - 1) / main.bm * per_row;
        const long long m1 = (tiles / slots) * slots / per_row * main.bm;
        if (m1 <= 0 || m1 >= m) continue;
        const double head = model_us(main, kind, m1, n, k, cus) + kSecondLaunchUs;
        for (const TileModel& rest : kTileModels) {
            if (rest.cfg == main.cfg || n % rest.bn != 0) continue;
            const double tr = head + model_us(rest, kind, m - m1, n, k, cus);
            if (tr < best_us) {
                best_us = tr;
                best = {main.cfg, static_cast<int>(m1), rest.cfg};
            }
        }
    }
    return best;
}

hipError_t launch_gemm_plan(const GemmPlan& p, const uint16_t* x, const uint16_t* w, const float* bias,
                            Residual res, int m, int n, int k, int epi, void* out, hipStream_t st) {
    constexpr int kGroupM = 8;
    ELIS_TRY(launch_gemm_config(p.main, p.main == 1 ? 1 : kGroupM, x, w, bias, res, p.m1, n, k, epi, out, st));
    if (p.m1 >= m) return hipSuccess;
    const size_t r0 = static_cast<size_t>(p.m1);
    const bool f32out = epi == ELIS_EPI_BIAS_RES_F32 || kResLnCode(epi);
    Residual rr = res;
    if (rr.x) rr.x += r0 * n;
    if (rr.stats) rr.stats += r0;
    void* o2 = f32out ? static_cast<void*>(static_cast<float*>(out) + r0 * n)
                      : static_cast<void*>(static_cast<uint16_t*>(out) + r0 * n);
    return launch_gemm_config(p.rest, kGroupM, x + r0 * k, w, bias, rr, m - p.m1, n, k, epi, o2, st);
}

// Every 32 x 32 x 16 configuration accumulates each output element in the same order with the
// same MFMA instruction and applies the same epilogue arithmetic, so neither the plan nor the
// split ever changes a result.
hipError_t launch_gemm(const uint16_t* x, const uint16_t* w, const float* bias, Residual res, int m, int n,
                       int k, int epi, void* out, hipStream_t st) {
    if (m < 1 || n % 64 != 0 || k % kBK != 0 || n < 64 || k < kBK) return hipErrorInvalidValue;
    return launch_gemm_plan(plan_gemm(m, n, k, epi), x, w, bias, res, m, n, k, epi, out, st);
}

}  // namespace elis
