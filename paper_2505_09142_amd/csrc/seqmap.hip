// Sequence map: validates the packed-batch boundaries and builds the table the
// other kernels index through. Every entry is clamped so that any later access
// stays inside [0, total) even when cu_seqlens is malformed.
#include "kernels.h"

namespace elis {

namespace {

constexpr int kThreads = 1024;

__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int u = __shfl_up(v, o, kWave);
        if (lane >= o) v += u;
    }
    return v;
}

__global__ __launch_bounds__(kThreads) void seqmap_kernel(const int32_t* __restrict__ cu, int n, int total,
                                                          int max_seqlen, int32_t* __restrict__ start,
                                                          int32_t* __restrict__ len,
                                                          int32_t* __restrict__ tile_off,
                                                          uint32_t* __restrict__ status) {
    __shared__ int wave_tot[kThreads / kWave];
    __shared__ int carry_s;
    __shared__ uint32_t flags_s;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    if (tid == 0) {
        carry_s = 0;
        flags_s = 0;
    }
    __syncthreads();
    uint32_t flags = 0;
    const int max_len = max_seqlen < total ? max_seqlen : total;
    for (int base = 0; base < n; base += kThreads) {
        const int s = base + tid;
        int tiles = 0;
        if (s < n) {
            int a = cu[s], b = cu[s + 1];
            if (s == 0 && a != 0) flags |= ELIS_DEV_BAD_CU;
            if (s == n - 1 && b != total) flags |= ELIS_DEV_BAD_CU;
            int L = b - a;
            if (L < 1) flags |= ELIS_DEV_BAD_CU;
            if (L > max_seqlen) flags |= ELIS_DEV_LONG_SEQ;
            L = L < 1 ? 1 : (L > max_len ? max_len : L);
            a = a < 0 ? 0 : (a > total - L ? total - L : a);
            start[s] = a;
            len[s] = L;
            tiles = (L + kAttnRowsPerBlock - 1) / kAttnRowsPerBlock;
        }
        const int incl = wave_incl_scan(tiles, lane);
        if (lane == kWave - 1) wave_tot[wid] = incl;
        __syncthreads();
        int wave_base = 0;
        for (int w = 0; w < wid; ++w) wave_base += wave_tot[w];
        const int carry = carry_s;
        if (s < n) tile_off[s] = carry + wave_base + incl - tiles;
        __syncthreads();
        if (tid == kThreads - 1) carry_s = carry + wave_base + incl;
        __syncthreads();
    }
    if (flags) atomicOr(&flags_s, flags);
    __syncthreads();
    if (tid == 0) {
        tile_off[n] = carry_s;
        *status = flags_s;
    }
}

}  // namespace

hipError_t launch_seqmap(const int32_t* cu, int n, int total, int max_seqlen, SeqTable tab, uint32_t* status,
                         hipStream_t st) {
    ELIS_TRY(launch_kernel(seqmap_kernel, dim3(1), dim3(kThreads), 0, st, cu, n, total, max_seqlen, tab.start,
                       tab.len, tab.tile_off, status));
    return hipSuccess;
}

}  // namespace elis
