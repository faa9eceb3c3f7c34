// Pooling + regression head: one work-group per sequence.
//
// CLS pooling takes the sequence's first final hidden vector (Sec. 3.2);
// mean pooling averages all of them, the CLS position included (Sec. 4.2).
// The head is linear d->1 or d->hidden->ReLU->1, computed in fp32; the result
// is mapped to tokens as shift + scale * y.
#include "kernels.h"

namespace elis {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxD = 2048;
constexpr int kMaxHidden = 4096;

__device__ __forceinline__ float block_sum(float v, float* red) {
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[wid] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kThreads / kWave; ++w) t += red[w];
    return t;
}

__global__ __launch_bounds__(kThreads) void pool_head_kernel(
    const float* __restrict__ hidden, const int32_t* __restrict__ start, const int32_t* __restrict__ len, int d,
    int pooling, int hh, const float* __restrict__ w1, const float* __restrict__ b1, const float* __restrict__ w2,
    const float* __restrict__ b2, float scale, float shift, float* __restrict__ out) {
    __shared__ float z[kMaxD];
    __shared__ float hid[kMaxHidden];
    __shared__ float red[kThreads / kWave];
    const int s = blockIdx.x, tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    const int a = start[s], L = len[s];
    const float* h0 = hidden + static_cast<size_t>(a) * d;
    if (pooling == ELIS_POOL_CLS) {
        for (int c = tid; c < d; c += kThreads) z[c] = h0[c];
    } else {
        const float inv = 1.0f / static_cast<float>(L);
        for (int c = tid; c < d; c += kThreads) {
            float acc = 0.f;
            for (int r = 0; r < L; ++r) acc += h0[static_cast<size_t>(r) * d + c];
            z[c] = acc * inv;
        }
    }
    __syncthreads();
    float part = 0.f;
    if (hh > 0) {
        for (int j = wid; j < hh; j += kThreads / kWave) {
            const float* wr = w1 + static_cast<size_t>(j) * d;
            float acc = 0.f;
            for (int c = lane; c < d; c += kWave) acc += wr[c] * z[c];
            acc = wave_sum(acc);
            if (lane == 0) hid[j] = fmaxf(acc + b1[j], 0.f);
        }
        __syncthreads();
        for (int j = tid; j < hh; j += kThreads) part += hid[j] * w2[j];
    } else {
        for (int c = tid; c < d; c += kThreads) part += z[c] * w2[c];
    }
    const float y = block_sum(part, red) + b2[0];
    if (tid == 0) out[s] = shift + scale * y;
}

}  // namespace

hipError_t launch_pool_head(const float* hidden, SeqTable tab, int n, int d, int pooling, int head_hidden,
                            const float* w1, const float* b1, const float* w2, const float* b2, float scale,
                            float shift, float* out, hipStream_t st) {
    if (d > kMaxD || head_hidden > kMaxHidden) return hipErrorInvalidValue;
    hipLaunchKernelGGL(pool_head_kernel, dim3(n), dim3(kThreads), 0, st, hidden, tab.start, tab.len, d, pooling,
                       head_hidden, w1, b1, w2, b2, scale, shift, out);
    return hipGetLastError();
}

}  // namespace elis
