// Sequence map: validates the packed-batch boundaries and builds the table the
// other kernels index through. Every entry is clamped so that any later access
// stays inside [0, total) even when cu_seqlens is malformed.
//
// Attention work list. The attention launch runs one work-group per (query tile,
// head), and a work-group's time grows with its sequence's length. Dispatched in
// batch order, the longest sequences' work-groups often start last and the kernel
// ends in a long, thinly occupied tail. The list therefore orders the query tiles
// longest sequence first (a counting sort on the number of 64-key tiles, lengths
// above 64 such tiles sharing the top bucket; batch order within a bucket), and
// each entry carries the tile's sequence start, length and first query, so a
// work-group reads its whole assignment with one load; slots past the list's end
// hold length 0, and their work-groups exit.
#include "kernels.h"

namespace elis {

namespace {

constexpr int kThreads = 1024;
constexpr int kBuckets = 64;  // sort key: 64-key tiles per sequence, capped
static_assert(kBuckets == kWave, "one bucket per lane in the per-wave bucket totals");

__device__ __forceinline__ int len_bucket(int L) {
    const int t = (L + 63) / 64;
    return t < kBuckets ? t - 1 : kBuckets - 1;
}

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
                                                          int32_t* __restrict__ work, int work_cap,
                                                          uint32_t* __restrict__ status) {
    __shared__ int wave_tot[kThreads / kWave];
    __shared__ int carry_s;
    __shared__ uint32_t flags_s;
    __shared__ int hist[kBuckets];          // query tiles per length bucket
    __shared__ int bucket_base[kBuckets];   // first list entry of each bucket
    __shared__ int bucket_carry[kBuckets];  // entries of the bucket taken by earlier chunks
    __shared__ int wave_b[kThreads / kWave][kBuckets];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    if (tid == 0) {
        carry_s = 0;
        flags_s = 0;
    }
    if (tid < kBuckets) {
        hist[tid] = 0;
        bucket_carry[tid] = 0;
    }
    __syncthreads();
    uint32_t flags = 0;
    const int max_len = max_seqlen < total ? max_seqlen : total;
    int a_first = 0, len_first = 0;  // this thread's entry of the first chunk, kept for the work list
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
            if (base == 0) {
                a_first = a;
                len_first = L;
            }
            tiles = (L + kAttnRowsPerBlock - 1) / kAttnRowsPerBlock;
            if (work) atomicAdd(&hist[len_bucket(L)], tiles);
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
    if (!work) return;  // uniform
    for (int idx = carry_s + tid; idx < work_cap; idx += kThreads)  // unused slots: length 0
        *reinterpret_cast<int4*>(work + 4 * static_cast<size_t>(idx)) = make_int4(0, 0, 0, 0);
    if (wid == 0) {  // bucket bases, longest bucket first: lane l scans bucket kBuckets - 1 - l
        const int c = hist[kBuckets - 1 - lane];
        bucket_base[kBuckets - 1 - lane] = wave_incl_scan(c, lane) - c;
    }
    __syncthreads();
    for (int base = 0; base < n; base += kThreads) {
        const int s = base + tid;
        int b = -1, tiles = 0, a = 0, L = 0;
        if (s < n) {  // this thread wrote start[s] and len[s] above
            a = base == 0 ? a_first : start[s];
            L = base == 0 ? len_first : len[s];
            tiles = (L + kAttnRowsPerBlock - 1) / kAttnRowsPerBlock;
            b = len_bucket(L);
        }
        // Entries of earlier sequences of the same bucket in this wave, and (lane l) the
        // wave's entries in bucket l; only the wave's lanes that hold a sequence are visited.
        int off = 0, lane_bucket_tot = 0;
        const int wave_seqs = n - base - wid * kWave;
        const int nv = wave_seqs < 0 ? 0 : (wave_seqs < kWave ? wave_seqs : kWave);
        for (int o = 0; o < nv; ++o) {
            const int ob = __builtin_amdgcn_readlane(b, o), ot = __builtin_amdgcn_readlane(tiles, o);
            off += (o < lane && ob == b) ? ot : 0;
            lane_bucket_tot += ob == lane ? ot : 0;
        }
        wave_b[wid][lane] = lane_bucket_tot;
        __syncthreads();
        if (s < n) {
            int first = bucket_base[b] + bucket_carry[b] + off;
            for (int w = 0; w < wid; ++w) first += wave_b[w][b];
            for (int q = 0; q < tiles; ++q) {
                const int idx = first + q;
                if (idx < work_cap)
                    *reinterpret_cast<int4*>(work + 4 * static_cast<size_t>(idx)) =
                        make_int4(a, L, q * kAttnRowsPerBlock, s);
            }
        }
        __syncthreads();
        if (tid < kBuckets) {
            int t = 0;
            for (int w = 0; w < kThreads / kWave; ++w) t += wave_b[w][tid];
            bucket_carry[tid] += t;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_seqmap(const int32_t* cu, int n, int total, int max_seqlen, SeqTable tab, uint32_t* status,
                         hipStream_t st) {
    ELIS_TRY(launch_kernel(seqmap_kernel, dim3(1), dim3(kThreads), 0, st, cu, n, total, max_seqlen, tab.start,
                       tab.len, tab.tile_off, tab.work, attn_work_capacity(n, total), status));
    return hipSuccess;
}

}  // namespace elis
