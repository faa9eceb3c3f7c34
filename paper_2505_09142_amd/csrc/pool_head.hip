// Pooling + regression head.
//
// CLS pooling takes the sequence's first final hidden vector (Sec. 3.2); mean
// pooling averages all of them, the CLS position included (Sec. 4.2). The head
// is linear d->1 or d->hidden->ReLU->1 in fp32; the result is mapped to tokens
// as shift + scale * y.
//
// Kernels (all reductions in a fixed order, so results are bitwise
// reproducible and independent of how sequences are packed):
//   pool_partial  mean pooling only: per (sequence, 256-column block, 64-row
//                 chunk) column sums, fully coalesced row reads;
//   pool_reduce   mean pooling only: chunk sums in order, divided by the length;
//   head_hidden   MLP head only: one wave per (hidden unit, 4 sequences), lanes
//                 across d, so each weight row is read once per 4 sequences;
//   head_out      one wave per sequence: ReLU(hidden + b1) . w2 + b2 (or z . w
//                 + b for the linear head), then shift + scale * y.
// For CLS pooling the head reads the CLS row of the hidden states in place.
#include "kernels.h"

namespace elis {

namespace {

constexpr int kCols = 256;      // columns per pooling work-group
constexpr int kSeqPerWave = 4;  // sequences sharing one weight-row read in head_hidden

__global__ __launch_bounds__(kCols) void pool_partial_kernel(const float* __restrict__ hidden,
                                                             const int32_t* __restrict__ start,
                                                             const int32_t* __restrict__ len, int d, int nchunk,
                                                             float* __restrict__ partial) {
    const int s = blockIdx.x, c = blockIdx.y * kCols + threadIdx.x, ch = blockIdx.z;
    if (c >= d) return;
    const int L = len[s];
    const int r0 = ch * kPoolChunk;
    float acc = 0.f;
    if (r0 < L) {
        const int r1 = (r0 + kPoolChunk < L) ? r0 + kPoolChunk : L;
        const float* h = hidden + (static_cast<size_t>(start[s]) + r0) * d + c;
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
        int r = r0;
        for (; r + 4 <= r1; r += 4, h += 4 * static_cast<size_t>(d)) {
            a0 += h[0];
            a1 += h[d];
            a2 += h[2 * static_cast<size_t>(d)];
            a3 += h[3 * static_cast<size_t>(d)];
        }
        for (; r < r1; ++r, h += d) a0 += h[0];
        acc = (a0 + a1) + (a2 + a3);
    }
    partial[(static_cast<size_t>(s) * nchunk + ch) * d + c] = acc;
}

__global__ __launch_bounds__(kCols) void pool_reduce_kernel(const float* __restrict__ partial,
                                                            const int32_t* __restrict__ len, int d, int nchunk,
                                                            float* __restrict__ z) {
    const int s = blockIdx.x, c = blockIdx.y * kCols + threadIdx.x;
    if (c >= d) return;
    const int L = len[s];
    const int used = (L + kPoolChunk - 1) / kPoolChunk;
    const float* p = partial + static_cast<size_t>(s) * nchunk * d + c;
    float acc = 0.f;
    for (int ch = 0; ch < used && ch < nchunk; ++ch) acc += p[static_cast<size_t>(ch) * d];
    z[static_cast<size_t>(s) * d + c] = acc / static_cast<float>(L);
}

__device__ __forceinline__ const float* pooled_row(int s, int pooling, const float* hidden, const float* z,
                                                   const int32_t* start, int d) {
    return pooling == ELIS_POOL_CLS ? hidden + static_cast<size_t>(start[s]) * d : z + static_cast<size_t>(s) * d;
}

// grid (hh, ceil(n / kSeqPerWave)), one wave per work-group.
__global__ __launch_bounds__(kWave) void head_hidden_kernel(const float* __restrict__ hidden,
                                                            const float* __restrict__ z,
                                                            const int32_t* __restrict__ start, int n, int d,
                                                            int pooling, int hh, const float* __restrict__ w1,
                                                            const float* __restrict__ b1,
                                                            float* __restrict__ hid) {
    const int j = blockIdx.x, s0 = blockIdx.y * kSeqPerWave, lane = threadIdx.x;
    const float* wr = w1 + static_cast<size_t>(j) * d;
    const float* zr[kSeqPerWave];
#pragma unroll
    for (int q = 0; q < kSeqPerWave; ++q)
        zr[q] = pooled_row(s0 + q < n ? s0 + q : n - 1, pooling, hidden, z, start, d);
    float acc[kSeqPerWave] = {0.f, 0.f, 0.f, 0.f};
    for (int c = 4 * lane; c < d; c += 4 * kWave) {
        const f32x4 w = *reinterpret_cast<const f32x4*>(wr + c);
#pragma unroll
        for (int q = 0; q < kSeqPerWave; ++q) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(zr[q] + c);
            acc[q] += (w[0] * v[0] + w[1] * v[1]) + (w[2] * v[2] + w[3] * v[3]);
        }
    }
#pragma unroll
    for (int q = 0; q < kSeqPerWave; ++q) {
        const float t = wave_sum(acc[q]);
        if (lane == 0 && s0 + q < n) hid[static_cast<size_t>(s0 + q) * hh + j] = fmaxf(t + b1[j], 0.f);
    }
}

// grid (n), one wave per work-group.
__global__ __launch_bounds__(kWave) void head_out_kernel(const float* __restrict__ hidden,
                                                         const float* __restrict__ z,
                                                         const int32_t* __restrict__ start, int d, int pooling,
                                                         int hh, const float* __restrict__ hid,
                                                         const float* __restrict__ w2, const float* __restrict__ b2,
                                                         float scale, float shift, float* __restrict__ out) {
    const int s = blockIdx.x, lane = threadIdx.x;
    const float* x = hh > 0 ? hid + static_cast<size_t>(s) * hh : pooled_row(s, pooling, hidden, z, start, d);
    const int len = hh > 0 ? hh : d;
    float acc = 0.f;
    for (int c = lane; c < len; c += kWave) acc += x[c] * w2[c];
    const float y = wave_sum(acc) + b2[0];
    if (lane == 0) out[s] = shift + scale * y;
}

}  // namespace

hipError_t launch_pool_head(const float* hidden, SeqTable tab, int n, int d, int pooling, int head_hidden,
                            const float* w1, const float* b1, const float* w2, const float* b2, float scale,
                            float shift, float* out, PoolScratch scr, hipStream_t st) {
    if (d % 4 != 0) return hipErrorInvalidValue;
    const dim3 cols(n, (d + kCols - 1) / kCols);
    if (pooling == ELIS_POOL_MEAN) {
        hipLaunchKernelGGL(pool_partial_kernel, dim3(n, cols.y, scr.nchunk), dim3(kCols), 0, st, hidden, tab.start,
                           tab.len, d, scr.nchunk, scr.partial);
        hipLaunchKernelGGL(pool_reduce_kernel, cols, dim3(kCols), 0, st, scr.partial, tab.len, d, scr.nchunk, scr.z);
    }
    if (head_hidden > 0)
        hipLaunchKernelGGL(head_hidden_kernel, dim3(head_hidden, (n + kSeqPerWave - 1) / kSeqPerWave), dim3(kWave), 0,
                           st, hidden, scr.z, tab.start, n, d, pooling, head_hidden, w1, b1, scr.hid);
    hipLaunchKernelGGL(head_out_kernel, dim3(n), dim3(kWave), 0, st, hidden, scr.z, tab.start, d, pooling, head_hidden,
                       scr.hid, w2, b2, scale, shift, out);
    return hipGetLastError();
}

}  // namespace elis
