// Row-wise kernels bound by HBM bandwidth: the fused embedding + LayerNorm and
// the LayerNorm that closes each post-LN sub-block.
//
// One wave per row; each lane owns float4 groups at columns 4*(lane + 64*i),
// so a wave reads a row in fully coalesced 1 KiB sweeps. Mean and variance are
// two-pass over the registers (no E[x^2] - E[x]^2 cancellation), reduced with
// cross-lane shuffles.
//
// Outputs (LnOut): the fp32 and/or bf16 normalised row, and optionally the row
// statistics (mean, rstd) instead of an fp32 copy: the fp32-output GEMM that
// consumes the row as its residual rebuilds y = fmaf((z - mean) * rstd, g, b)
// from the pre-norm row z, which saves writing and re-reading an fp32 copy.
// Floating-point contraction is off in the row finish: every product and sum is
// rounded as written (only the explicit fmaf is fused), so the normalised row it
// writes is exactly what that rebuild computes from the stored mean and rstd (with
// contraction the compiler fused the mean into z - mean and the variance into
// var + eps, and the two sides could differ in the last bit).
#include "kernels.h"

namespace elis {

namespace {

constexpr int kRowsPerBlock = 4;  // 4 waves, one row each

template <int VPL>
__device__ __forceinline__ void ln_finish(f32x4 (&v)[VPL], int lane, int d, const float* __restrict__ g,
                                          const float* __restrict__ b, float eps, size_t row, const LnOut& o) {
#pragma clang fp contract(off)
    float* o32 = o.y32 ? o.y32 + row * d : nullptr;
    uint16_t* o16 = o.y16 ? o.y16 + row * d : nullptr;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int e = 4 * (lane + kWave * i);
        if (e < d) s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
    }
    const float inv_d = 1.0f / static_cast<float>(d);
    const float mean = wave_sum(s) * inv_d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int e = 4 * (lane + kWave * i);
        if (e < d) {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float t = v[i][c] - mean;
                q += t * t;
            }
        }
    }
    const float var = wave_sum(q) * inv_d;
    const float rstd = 1.0f / sqrtf(var + eps);
    if (o.stats && lane == 0) o.stats[row] = make_float2(mean, rstd);
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int e = 4 * (lane + kWave * i);
        if (e < d) {
            const f32x4 gv = *reinterpret_cast<const f32x4*>(g + e);
            const f32x4 bv = *reinterpret_cast<const f32x4*>(b + e);
            f32x4 y;
#pragma unroll
            for (int c = 0; c < 4; ++c) y[c] = fmaf((v[i][c] - mean) * rstd, gv[c], bv[c]);
            if (o32) *reinterpret_cast<f32x4*>(o32 + e) = y;
            if (o16) {
                u32x2 p;
                p[0] = pack_bf16x2(y[0], y[1]);
                p[1] = pack_bf16x2(y[2], y[3]);
                *reinterpret_cast<u32x2*>(o16 + e) = p;
            }
        }
    }
}

__device__ __forceinline__ f32x4 load_bf16x4(const uint16_t* p) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
    f32x4 r;
    r[0] = __uint_as_float(w[0] << 16);
    r[1] = __uint_as_float(w[0] & 0xffff0000u);
    r[2] = __uint_as_float(w[1] << 16);
    r[3] = __uint_as_float(w[1] & 0xffff0000u);
    return r;
}

template <int VPL>
__global__ __launch_bounds__(kRowsPerBlock* kWave) void embed_ln_kernel(
    const int32_t* __restrict__ ids, const int32_t* __restrict__ cu, int n, int total,
    const uint16_t* __restrict__ word, const uint16_t* __restrict__ pos, const float* __restrict__ type0,
    const float* __restrict__ g, const float* __restrict__ b, int d, int vocab, int max_pos, float eps,
    LnOut out, uint32_t* __restrict__ status) {
    const int lane = threadIdx.x & (kWave - 1);
    const int t = blockIdx.x * kRowsPerBlock + (threadIdx.x / kWave);
    // Up to 255 sequences, the segment search runs over a copy of cu in LDS (one load per
    // thread, then LDS latency per search step instead of a dependent global load).
    __shared__ int32_t cu_s[kRowsPerBlock * kWave];
    const bool staged = n < kRowsPerBlock * kWave;  // n + 1 entries fit; uniform
    if (staged) {
        for (int i = threadIdx.x; i <= n; i += kRowsPerBlock * kWave) cu_s[i] = cu[i];
        __syncthreads();
    }
    if (t >= total) return;
    const int s = staged ? find_segment(cu_s, n, t) : find_segment(cu, n, t);
    int p = t - (staged ? cu_s[s] : cu[s]);
    p = p < 0 ? 0 : (p >= max_pos ? max_pos - 1 : p);
    int id = ids[t];
    if (id < 0 || id >= vocab) {
        if (lane == 0) atomicOr(status, ELIS_DEV_BAD_TOKEN);
        id = id < 0 ? 0 : vocab - 1;
    }
    const uint16_t* wr = word + static_cast<size_t>(id) * d;
    const uint16_t* pr = pos + static_cast<size_t>(p) * d;
    f32x4 v[VPL];
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int e = 4 * (lane + kWave * i);
        if (e < d) {
            v[i] = load_bf16x4(wr + e) + load_bf16x4(pr + e) + *reinterpret_cast<const f32x4*>(type0 + e);
            if (out.z32) *reinterpret_cast<f32x4*>(out.z32 + static_cast<size_t>(t) * d + e) = v[i];
        }
    }
    ln_finish<VPL>(v, lane, d, g, b, eps, static_cast<size_t>(t), out);
}

template <int VPL>
__global__ __launch_bounds__(kRowsPerBlock* kWave) void layernorm_kernel(const float* __restrict__ x,
                                                                         const float* __restrict__ g,
                                                                         const float* __restrict__ b, int rows,
                                                                         int d, float eps, LnOut out) {
    const int lane = threadIdx.x & (kWave - 1);
    const int r = blockIdx.x * kRowsPerBlock + (threadIdx.x / kWave);
    if (r >= rows) return;
    const size_t off = static_cast<size_t>(r) * d;
    f32x4 v[VPL];
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
        const int e = 4 * (lane + kWave * i);
        if (e < d) v[i] = *reinterpret_cast<const f32x4*>(x + off + e);
    }
    ln_finish<VPL>(v, lane, d, g, b, eps, static_cast<size_t>(r), out);
}

// One wave per gathered row: float4 lanes across the row, lane 0 also copies the statistics.
__global__ __launch_bounds__(kRowsPerBlock* kWave) void gather_rows_kernel(
    const float* __restrict__ src, const float2* __restrict__ src_stats, const int32_t* __restrict__ start, int n,
    int d, float* __restrict__ dst, float2* __restrict__ dst_stats) {
    const int lane = threadIdx.x & (kWave - 1);
    const int s = blockIdx.x * kRowsPerBlock + (threadIdx.x / kWave);
    if (s >= n) return;
    const size_t from = static_cast<size_t>(start[s]) * d, to = static_cast<size_t>(s) * d;
    for (int e = 4 * lane; e < d; e += 4 * kWave)
        *reinterpret_cast<f32x4*>(dst + to + e) = *reinterpret_cast<const f32x4*>(src + from + e);
    if (lane == 0) dst_stats[s] = src_stats[start[s]];
}

}  // namespace

hipError_t launch_gather_rows(const float* src, const float2* src_stats, const int32_t* start, int n, int d,
                              float* dst, float2* dst_stats, hipStream_t st) {
    if (n < 1 || d % 4 != 0) return hipErrorInvalidValue;
    ELIS_TRY(launch_kernel(gather_rows_kernel, dim3((n + kRowsPerBlock - 1) / kRowsPerBlock),
                           dim3(kRowsPerBlock * kWave), 0, st, src, src_stats, start, n, d, dst, dst_stats));
    return hipSuccess;
}

#define ELIS_VPL_SWITCH(d, CALL)          \
    switch ((d + 255) / 256) {            \
        case 1: CALL(1); break;           \
        case 2: CALL(2); break;           \
        case 3: CALL(3); break;           \
        case 4: CALL(4); break;           \
        case 5: CALL(5); break;           \
        case 6: CALL(6); break;           \
        case 7: CALL(7); break;           \
        case 8: CALL(8); break;           \
        default: return hipErrorInvalidValue; \
    }

hipError_t launch_embed_ln(const int32_t* ids, const int32_t* cu, int n, int total, const uint16_t* word,
                           const uint16_t* pos, const float* type0, const float* g, const float* b, int d,
                           int vocab, int max_pos, float eps, LnOut out, uint32_t* status, hipStream_t st) {
    const dim3 grid((total + kRowsPerBlock - 1) / kRowsPerBlock), block(kRowsPerBlock * kWave);
#define CALL(V)                                                                                          \
    ELIS_TRY(launch_kernel(embed_ln_kernel<V>, grid, block, 0, st, ids, cu, n, total, word, pos, type0, g, b, d, \
                       vocab, max_pos, eps, out, status))
    ELIS_VPL_SWITCH(d, CALL)
#undef CALL
    return hipSuccess;
}

hipError_t launch_layernorm(const float* x, const float* g, const float* b, int rows, int d, float eps,
                            LnOut out, hipStream_t st) {
    const dim3 grid((rows + kRowsPerBlock - 1) / kRowsPerBlock), block(kRowsPerBlock * kWave);
#define CALL(V) ELIS_TRY(launch_kernel(layernorm_kernel<V>, grid, block, 0, st, x, g, b, rows, d, eps, out))
    ELIS_VPL_SWITCH(d, CALL)
#undef CALL
    return hipSuccess;
}

}  // namespace elis
