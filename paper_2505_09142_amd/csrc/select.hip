// ISRTF batch selection on the device (Sec. 4.1: the batch is formed from the
// jobs with the fewest predicted remaining tokens; ties go to the earlier
// arrival, then the lower index).
//
// Each job gets a total-order key (orderable-u32(pred), arrival, index):
//   * the float is mapped to an unsigned integer whose order is the float
//     order, with -0 folded onto +0 and every NaN mapped to the maximum (after
//     +inf), so the comparison is exact integer work with no rounding;
//   * n <= 1024: one work-group ranks every key by counting the keys below it
//     (keys in LDS, read as broadcasts), and the job of rank r < k lands in
//     out_idx[r];
//   * 1024 < n <= 8192: one work-group bitonic-sorts the keys in LDS (padded
//     to a power of two with +max sentinels) and writes the first k.
#include <limits.h>

#include "kernels.h"

namespace elis {

namespace {

constexpr int kThreads = 1024;
constexpr int kRankMaxN = 1024;
constexpr int kSortMaxN = 8192;

__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0xffffffffu;  // NaN, any sign / payload
    if (u == 0x80000000u) u = 0u;                               // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ bool key_less(uint32_t ka, int64_t aa, int ia, uint32_t kb, int64_t ab, int ib) {
    if (ka != kb) return ka < kb;
    if (aa != ab) return aa < ab;
    return ia < ib;
}

__global__ __launch_bounds__(kThreads) void select_rank_kernel(const float* __restrict__ pred,
                                                               const int64_t* __restrict__ arrival, int n, int k,
                                                               int32_t* __restrict__ out_idx,
                                                               int32_t* __restrict__ out_count,
                                                               uint32_t* __restrict__ status) {
    __shared__ uint32_t sk[kRankMaxN];
    __shared__ int64_t sa[kRankMaxN];
    const int i = threadIdx.x;
    if (i < n) {
        sk[i] = order_key(pred[i]);
        sa[i] = arrival[i];
    }
    __syncthreads();
    if (i < n) {
        const uint32_t ki = sk[i];
        const int64_t ai = sa[i];
        int rank = 0;
        for (int j = 0; j < n; ++j) rank += key_less(sk[j], sa[j], j, ki, ai, i) ? 1 : 0;
        if (rank < k) out_idx[rank] = i;
    }
    if (i == 0) {
        *out_count = k < n ? k : n;
        *status = 0u;
    }
}

__global__ __launch_bounds__(kThreads) void select_sort_kernel(const float* __restrict__ pred,
                                                               const int64_t* __restrict__ arrival, int n, int k,
                                                               int32_t* __restrict__ out_idx,
                                                               int32_t* __restrict__ out_count,
                                                               uint32_t* __restrict__ status) {
    __shared__ uint32_t sk[kSortMaxN];
    __shared__ int32_t si[kSortMaxN];
    __shared__ int64_t sa[kSortMaxN];
    int P = 1;
    while (P < n) P <<= 1;
    for (int i = threadIdx.x; i < P; i += kThreads) {
        if (i < n) {
            sk[i] = order_key(pred[i]);
            sa[i] = arrival[i];
            si[i] = i;
        } else {
            sk[i] = 0xffffffffu;
            sa[i] = LLONG_MAX;
            si[i] = INT_MAX;
        }
    }
    __syncthreads();
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = threadIdx.x; t < (P >> 1); t += kThreads) {
                const int lo = 2 * t - (t & (stride - 1));
                const int hi = lo + stride;
                const bool up = (lo & size) == 0;
                const bool hi_first = key_less(sk[hi], sa[hi], si[hi], sk[lo], sa[lo], si[lo]);
                if (hi_first == up) {
                    const uint32_t tk = sk[lo];
                    sk[lo] = sk[hi];
                    sk[hi] = tk;
                    const int64_t ta = sa[lo];
                    sa[lo] = sa[hi];
                    sa[hi] = ta;
                    const int32_t ti = si[lo];
                    si[lo] = si[hi];
                    si[hi] = ti;
                }
            }
            __syncthreads();
        }
    }
    const int m = k < n ? k : n;
    for (int r = threadIdx.x; r < m; r += kThreads) out_idx[r] = si[r];
    if (threadIdx.x == 0) {
        *out_count = m;
        *status = 0u;
    }
}

}  // namespace

int select_max_n() { return kSortMaxN; }

hipError_t launch_select(const float* pred, const int64_t* arrival, int n, int k, int32_t* out_idx,
                         int32_t* out_count, uint32_t* status, hipStream_t st) {
    if (n < 1 || n > kSortMaxN || k < 0) return hipErrorInvalidValue;
    if (n <= kRankMaxN)
        hipLaunchKernelGGL(select_rank_kernel, dim3(1), dim3(kThreads), 0, st, pred, arrival, n, k, out_idx, out_count,
                           status);
    else
        hipLaunchKernelGGL(select_sort_kernel, dim3(1), dim3(kThreads), 0, st, pred, arrival, n, k, out_idx, out_count,
                           status);
    return hipGetLastError();
}

}  // namespace elis
