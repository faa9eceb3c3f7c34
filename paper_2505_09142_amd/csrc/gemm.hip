// Dense layers of the encoder on the CDNA4 matrix cores:
//   out[m, n] = epilogue( sum_k x[m, k] * w[n, k] + bias[n] )
// x is the activation, bf16 [M, K] row-major; w is the weight, bf16 [N, K]
// row-major ([out, in]); both operands are K-contiguous. fp32 accumulation.
//
// Tiling. A work-group computes a BM x BN tile with WM x WN waves; each wave
// owns a (BM/WM) x (BN/WN) sub-tile made of 16 x 16 MFMA blocks
// (v_mfma_f32_16x16x32_bf16: 16 x 16 output, 32-deep k per instruction).
// K advances in steps of 64 through two LDS stages: while the waves multiply
// out of one stage, the next k-slab is already in flight from HBM into
// registers and is written to the other stage afterwards (one barrier per
// k-step).
//
// LDS layout. A k-slab row is 64 bf16 = 128 bytes = eight 16-byte chunks; the
// chunk index is XOR-swizzled with the row (chunk ^ (row & 7)) so the 16 rows
// that one MFMA operand read touches fall on different banks.
//
// Operand order. The MFMA is issued as (weight fragment, activation
// fragment), which computes the transposed tile: lane l then holds 4
// consecutive output columns of one output row, so the epilogue reads
// bias / residual and writes the output as 16-byte (fp32) or 8-byte (bf16)
// vectors.
//
// Work-group order. The hardware hands consecutive work-group ids round-robin
// to the 8 XCDs (each with its own L2). Ids are remapped so every XCD gets one
// contiguous range of tiles, ordered N-fastest: the tiles an XCD runs together
// share their activation rows, which are then fetched from HBM once per XCD.
#include "kernels.h"

namespace elis {

namespace {

constexpr int kBK = 64;
// Same arithmetic as ELIS_EPI_BIAS_RES_F32; a separate instantiation so that the
// second feed-forward product shows up under its own kernel name in profiles.
constexpr int kEpiResF32Ffn2 = 3;

__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    constexpr int kXcd = 8;
    const int per = nblk / kXcd, rem = nblk % kXcd;
    const int xcd = bid % kXcd, local = bid / kXcd;
    return xcd * per + (xcd < rem ? xcd : rem) + local;
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM* WN* kWave) void gemm_kernel(const uint16_t* __restrict__ A,
                                                             const uint16_t* __restrict__ B,
                                                             const float* __restrict__ bias,
                                                             const float* __restrict__ res, void* __restrict__ out,
                                                             int M, int N, int K) {
    constexpr int NT = WM * WN * kWave;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 16, FN = TN / 16;
    constexpr int ACH = BM * 8 / NT, BCH = BN * 8 / NT;  // 16-byte chunks per thread per k-slab
    static_assert(BM * 8 % NT == 0 && BN * 8 % NT == 0, "tile must split evenly over the threads");
    static_assert(TM % 16 == 0 && TN % 16 == 0, "wave tile must be a multiple of 16");

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
    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

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

    const int r16 = lane & 15, kg = lane >> 4;
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT) gload((kt + 1) * kBK);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int c = ks * 4 + kg;
            bf16x8 af[FM], bfr[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const int row = wm * TM + i * 16 + r16;
                af[i] = *reinterpret_cast<const bf16x8*>(&sA[cur][row * kBK + ((c ^ (row & 7)) * 8)]);
            }
#pragma unroll
            for (int j = 0; j < FN; ++j) {
                const int row = wn * TN + j * 16 + r16;
                bfr[j] = *reinterpret_cast<const bf16x8*>(&sB[cur][row * kBK + ((c ^ (row & 7)) * 8)]);
            }
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < KT) sstore(cur ^ 1);
        __syncthreads();
    }

    // Epilogue: lane holds C[m][n .. n+3] for m = row r16 of block i, n = 4*kg in block j.
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = m0 + wm * TM + i * 16 + r16;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * TN + j * 16 + 4 * kg;
            f32x4 v = acc[i][j] + *reinterpret_cast<const f32x4*>(bias + n);
            const size_t o = static_cast<size_t>(m) * N + n;
            if constexpr (EPI == ELIS_EPI_BIAS_RES_F32 || EPI == kEpiResF32Ffn2) {
                v += *reinterpret_cast<const f32x4*>(res + o);
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

template <int BM, int BN, int WM, int WN>
hipError_t launch_tile(const uint16_t* x, const uint16_t* w, const float* bias, const float* res, int m, int n,
                       int k, int epi, void* out, hipStream_t st) {
    const dim3 grid(((m + BM - 1) / BM) * (n / BN)), block(WM * WN * kWave);
    switch (epi) {
        case ELIS_EPI_BIAS_BF16:
            hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, ELIS_EPI_BIAS_BF16>), grid, block, 0, st, x, w, bias,
                               res, out, m, n, k);
            break;
        case ELIS_EPI_BIAS_GELU_BF16:
            hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, ELIS_EPI_BIAS_GELU_BF16>), grid, block, 0, st, x, w,
                               bias, res, out, m, n, k);
            break;
        case ELIS_EPI_BIAS_RES_F32:
            hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, ELIS_EPI_BIAS_RES_F32>), grid, block, 0, st, x, w,
                               bias, res, out, m, n, k);
            break;
        case kEpiResF32Ffn2:
            hipLaunchKernelGGL((gemm_kernel<BM, BN, WM, WN, kEpiResF32Ffn2>), grid, block, 0, st, x, w, bias, res,
                               out, m, n, k);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const uint16_t* x, const uint16_t* w, const float* bias, const float* res, int m, int n,
                       int k, int epi, void* out, hipStream_t st, bool ffn2) {
    if (ffn2 && epi == ELIS_EPI_BIAS_RES_F32) epi = kEpiResF32Ffn2;
    if (m < 1 || n % 64 != 0 || k % kBK != 0 || n < 64 || k < kBK) return hipErrorInvalidValue;
    if (n % 128 == 0) return launch_tile<128, 128, 2, 2>(x, w, bias, res, m, n, k, epi, out, st);
    return launch_tile<128, 64, 2, 2>(x, w, bias, res, m, n, k, epi, out, st);
}

}  // namespace elis
