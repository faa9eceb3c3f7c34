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
//     to a power of two with +max sentinels) and writes the first k;
//   * larger n (k <= 8192): radix selection over the whole device, most
//     significant digit first. Three counting passes over the float keys
//     (11, 11, 10 bits) fix the key P of the k-th job: in every pass each
//     work-group histograms its own contiguous chunk of jobs (those matching
//     the prefix fixed so far) and stores the counts; 32 small work-groups
//     total the buckets and the last of them picks the bucket holding the
//     k-th job. A scatter pass then lists, per chunk and in index order, the
//     jobs with key < P and the ties (key == P). Nothing in these passes is a
//     same-address global atomic (those serialise at tens of ns apiece across
//     the XCDs). A single work-group finishes: it takes the needed number of
//     ties by (arrival, index) - an LDS sort when there are at most 8192 of
//     them, otherwise a radix selection of its own over the 96-bit
//     (arrival, index) keys - and sorts the k chosen jobs by the full key.
//     The pred array is read four times (16 bytes per job); arrivals are read
//     for ties only.
#include <limits.h>

#include <mutex>

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
        // rank = number of jobs ordered before job i (key, then arrival, then index), counted
        // without branches so the LDS reads of consecutive j overlap
        int rank = 0;
#pragma unroll 8
        for (int j = 0; j < n; ++j) {
            const uint32_t kj = sk[j];
            const int64_t aj = sa[j];
            rank += static_cast<int>((kj < ki) | ((kj == ki) & ((aj < ai) | ((aj == ai) & (j < i)))));
        }
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

// ------------------------------------------------------------------------------ large n
constexpr int kLargeMaxN = 1 << 28;
constexpr int kBins = 2048;        // 11-bit digits
constexpr int kBlock = 1024;       // threads of the counting / scatter work-groups
constexpr int kMaxGroups = 256;    // work-groups of a counting / scatter pass (one chunk each)
constexpr int kReduceBlocks = kBins / 64;  // 64 bins per reducing work-group

// Device state of one large selection (workspace, written by select_init_kernel).
struct SelState {
    uint32_t need;      // jobs still to choose inside the current prefix
    uint32_t level;     // leading key bits fixed so far (0, 11, 22, 32)
    uint32_t prefix;    // their value
    uint32_t resolved;  // the bucket of the current prefix is taken whole
    uint32_t ticket;    // reduce work-groups done with the current pass
    uint32_t pad[3];
};

struct LargeWs {
    uint32_t* status;
    SelState* state;
    uint32_t* totals;   // [kBins] bucket counts of the current pass
    uint32_t* partial;  // [groups][kBins] per-work-group counts of the current pass
    uint32_t* counts;   // [groups][2] jobs chosen / tied, per work-group
    int32_t* chosen;    // [groups][kSortMaxN] chosen indices, per work-group
    int32_t* ties;      // [n] tied indices, each work-group at the start of its own chunk
    int32_t* picked;    // [kSortMaxN] ties taken by (arrival, index)
    int chunk;          // jobs per work-group
    int groups;
};

__device__ __forceinline__ uint32_t ld_relaxed(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Four consecutive predictions i .. i+3 (16-byte load when aligned and in range); lanes past
// hi read nothing and get 0.
__device__ __forceinline__ void load4(const float* __restrict__ pred, int i, int hi, bool vec, float (&v)[4]) {
    if (vec && i + 3 < hi) {
        const f32x4 f = *reinterpret_cast<const f32x4*>(pred + i);
#pragma unroll
        for (int c = 0; c < 4; ++c) v[c] = f[c];
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) v[c] = (i + c < hi) ? pred[i + c] : 0.f;
    }
}

// Exclusive prefix over the wave of a per-lane count below 8, and the wave total.
__device__ __forceinline__ uint32_t wave_prefix8(uint32_t c, uint32_t& total) {
    uint32_t ex = 0;
    total = 0;
#pragma unroll
    for (int bit = 0; bit < 3; ++bit) {
        const uint64_t m = __builtin_amdgcn_ballot_w64((c >> bit) & 1u);
        ex += __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)) << bit;
        total += static_cast<uint32_t>(__builtin_popcountll(m)) << bit;
    }
    return ex;
}

__global__ __launch_bounds__(256) void select_init_kernel(LargeWs ws, int k, int32_t* __restrict__ out_count) {
    if (threadIdx.x == 0) {
        SelState s{};
        s.need = static_cast<uint32_t>(k);
        *ws.state = s;
        *ws.status = 0u;
        *out_count = k;
    }
}

// Counting pass over one chunk: histogram of digit (key >> SHIFT) & (2^BITS - 1) of the jobs
// whose leading key bits equal the current prefix, stored (not added) to partial[group].
template <int SHIFT, int BITS>
__global__ __launch_bounds__(kBlock) void select_count_kernel(const float* __restrict__ pred, int n, LargeWs ws) {
    __shared__ uint32_t lh[kBins];
    const SelState* st = ws.state;
    if (st->resolved) return;
    const uint32_t level = st->level, prefix = st->prefix;
    for (int b = threadIdx.x; b < kBins; b += kBlock) lh[b] = 0u;
    __syncthreads();
    const int lo = blockIdx.x * ws.chunk;
    const int hi = lo + ws.chunk < n ? lo + ws.chunk : n;
    const bool vec = (reinterpret_cast<uintptr_t>(pred) & 15u) == 0;
    for (int base = lo; base < hi; base += 4 * kBlock) {
        float v[4];
        load4(pred, base + 4 * threadIdx.x, hi, vec, v);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const bool in = base + 4 * static_cast<int>(threadIdx.x) + c < hi;
            const uint32_t key = order_key(v[c]);
            const bool take = in && (level == 0 || (key >> (32 - level)) == prefix);
            const uint32_t d = (key >> SHIFT) & ((1u << BITS) - 1u);
            // Plain per-lane LDS atomics: measured faster than aggregating equal digits of a
            // wave first, even for the few leading digits of real predictions.
            if (take) atomicAdd(&lh[d], 1u);
        }
    }
    __syncthreads();
    uint32_t* out = ws.partial + static_cast<size_t>(blockIdx.x) * kBins;
    for (int b = threadIdx.x; b < kBins; b += kBlock) out[b] = lh[b];
}

// Bucket totals over the work-groups: each of kReduceBlocks work-groups owns 64 bins, its
// threads split the chunks 16 ways; the last work-group to finish picks the bucket holding
// the need-th job and advances the state.
template <int BITS>
__global__ __launch_bounds__(1024) void select_reduce_kernel(LargeWs ws) {
    __shared__ uint32_t part[16][64];
    __shared__ uint32_t scan[256];
    __shared__ bool last;
    const SelState* st = ws.state;
    if (st->resolved) return;
    const int b = threadIdx.x & 63, slice = threadIdx.x >> 6;
    const int bin = blockIdx.x * 64 + b;
    uint32_t t = 0;
    const int groups = ws.groups;
#pragma unroll 16
    for (int g = slice; g < groups; g += 16) t += ws.partial[static_cast<size_t>(g) * kBins + bin];
    part[slice][b] = t;
    __syncthreads();
    if (threadIdx.x < 64) {
        uint32_t s2 = 0;
#pragma unroll
        for (int q = 0; q < 16; ++q) s2 += part[q][threadIdx.x];
        ws.totals[blockIdx.x * 64 + threadIdx.x] = s2;
    }
    // One release fence after the barrier covers the work-group's stores (fences are costly
    // here: an agent-scope fence writes back and invalidates the XCD's L2).
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        last = atomicAdd(&ws.state->ticket, 1u) == kReduceBlocks - 1;
        if (last) __threadfence();
    }
    __syncthreads();
    if (!last) return;  // uniform over the work-group
    // The first 256 threads scan 8 bins each; all 1024 take part in the barriers.
    constexpr int PER = kBins / 256;
    const bool act = threadIdx.x < 256;
    uint32_t h[PER], sum = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        h[j] = act ? ld_relaxed(&ws.totals[threadIdx.x * PER + j]) : 0u;
        sum += h[j];
    }
    if (act) scan[threadIdx.x] = sum;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const uint32_t v = (act && threadIdx.x >= off) ? scan[threadIdx.x - off] : 0u;
        __syncthreads();
        if (act) scan[threadIdx.x] += v;
        __syncthreads();
    }
    if (!act) return;
    const uint32_t need = st->need, level = st->level, prefix = st->prefix;
    uint32_t below = scan[threadIdx.x] - sum;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        if (below < need && need <= below + h[j]) {
            SelState* w = ws.state;
            w->prefix = (prefix << BITS) | static_cast<uint32_t>(threadIdx.x * PER + j);
            w->level = level + BITS;
            w->need = need - below;
            w->resolved = (h[j] == need - below) ? 1u : 0u;
            w->ticket = 0u;
        }
        below += h[j];
    }
}

// Scatter over one chunk, in index order: key < prefix (or == prefix when resolved) ->
// chosen[group]; key == prefix otherwise -> this chunk's part of the tie list.
__global__ __launch_bounds__(kBlock) void select_scatter_kernel(const float* __restrict__ pred, int n, LargeWs ws) {
    __shared__ uint32_t wsum[2][kBlock / kWave];
    const SelState* st = ws.state;
    const uint32_t level = st->level, prefix = st->prefix;
    const bool resolved = st->resolved != 0u;
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const int lo = blockIdx.x * ws.chunk;
    const int hi = lo + ws.chunk < n ? lo + ws.chunk : n;
    int32_t* chosen = ws.chosen + static_cast<size_t>(blockIdx.x) * kSortMaxN;
    int32_t* ties = ws.ties + lo;
    const bool vec = (reinterpret_cast<uintptr_t>(pred) & 15u) == 0;
    uint32_t nc = 0, nt = 0;  // running counts of this work-group (uniform)
    for (int base = lo; base < hi; base += 4 * kBlock) {
        const int i0 = base + 4 * threadIdx.x;
        float v[4];
        load4(pred, i0, hi, vec, v);
        bool c[4], t[4];
        uint32_t cc = 0, ct = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t top = order_key(v[q]) >> (32 - level);
            const bool in = i0 + q < hi;
            c[q] = in && (top < prefix || (top == prefix && resolved));
            t[q] = in && top == prefix && !resolved;
            cc += c[q] ? 1u : 0u;
            ct += t[q] ? 1u : 0u;
        }
        uint32_t wc, wt;
        const uint32_t rc = wave_prefix8(cc, wc), rt = wave_prefix8(ct, wt);
        if (lane == 0) {
            wsum[0][wv] = wc;
            wsum[1][wv] = wt;
        }
        __syncthreads();
        uint32_t oc = nc, ot = nt, tc = 0, tt = 0;
        for (int w = 0; w < kBlock / kWave; ++w) {
            if (w < wv) {
                oc += wsum[0][w];
                ot += wsum[1][w];
            }
            tc += wsum[0][w];
            tt += wsum[1][w];
        }
        oc += rc;
        ot += rt;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (c[q]) chosen[oc++] = i0 + q;
            if (t[q]) ties[ot++] = i0 + q;
        }
        nc += tc;
        nt += tt;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        ws.counts[2 * blockIdx.x] = nc;
        ws.counts[2 * blockIdx.x + 1] = nt;
    }
}

// 96-bit tie key (arrival made unsigned-orderable, then index): bits [lo, lo + w).
__device__ __forceinline__ uint32_t tie_digit(uint64_t a, uint32_t idx, int lo, int w) {
    const uint64_t mask = (1ull << w) - 1ull;
    if (lo >= 32) return static_cast<uint32_t>((a >> (lo - 32)) & mask);
    if (lo + w <= 32) return static_cast<uint32_t>((idx >> lo) & mask);
    return static_cast<uint32_t>((((a << (32 - lo)) | (idx >> lo))) & mask);
}

__device__ __forceinline__ uint64_t arrival_key(int64_t a) { return static_cast<uint64_t>(a) ^ 0x8000000000000000ull; }

// One work-group: bitonic sort of P (power of two) entries in LDS by (key, arrival, index).
__device__ void block_bitonic(uint32_t* sk, int64_t* sa, int32_t* si, int P) {
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
}

__device__ __forceinline__ int pow2_at_least(int n) {
    int P = 1;
    while (P < n) P <<= 1;
    return P;
}

// Exclusive scan of per-work-group counts (groups <= kThreads) into offs[g]; returns the total.
__device__ uint32_t block_offsets(const uint32_t* counts, int which, int groups, uint32_t* offs, uint32_t* scan) {
    const uint32_t v = threadIdx.x < groups ? counts[2 * threadIdx.x + which] : 0u;
    scan[threadIdx.x] = v;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        const uint32_t u = threadIdx.x >= off ? scan[threadIdx.x - off] : 0u;
        __syncthreads();
        scan[threadIdx.x] += u;
        __syncthreads();
    }
    if (threadIdx.x < groups) offs[threadIdx.x] = scan[threadIdx.x] - v;
    const uint32_t total = scan[kThreads - 1];
    __syncthreads();
    return total;
}

// Index r (< total) of a list split over work-groups: which group holds it (binary search
// over the exclusive offsets) and at which position.
__device__ __forceinline__ int find_group(const uint32_t* offs, int groups, uint32_t r) {
    int lo = 0, hi = groups - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (offs[mid] <= r) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// Final work-group: choose the needed ties by (arrival, index), then sort the k chosen jobs.
__global__ __launch_bounds__(kThreads) void select_final_kernel(const float* __restrict__ pred,
                                                                const int64_t* __restrict__ arrival, int k, LargeWs ws,
                                                                int32_t* __restrict__ out_idx) {
    __shared__ uint32_t sk[kSortMaxN];
    __shared__ int64_t sa[kSortMaxN];
    __shared__ int32_t si[kSortMaxN];
    __shared__ uint32_t offc[kMaxGroups], offt[kMaxGroups];
    __shared__ uint32_t scan[kThreads];
    __shared__ uint32_t hist[kBins];
    __shared__ uint32_t sh_bucket, sh_below, sh_cnt;
    const int groups = ws.groups;
    const uint32_t nchosen = block_offsets(ws.counts, 0, groups, offc, scan);
    uint32_t ntie = block_offsets(ws.counts, 1, groups, offt, scan);
    const uint32_t need0 = ws.state->resolved ? 0u : ws.state->need;
    uint32_t npicked = 0;
    if (need0 > 0 && ntie <= static_cast<uint32_t>(kSortMaxN)) {
        // All ties share the float key: sort them by (arrival, index), take the first need0.
        const int P = pow2_at_least(static_cast<int>(ntie));
        for (int r = threadIdx.x; r < P; r += kThreads) {
            if (r < static_cast<int>(ntie)) {
                const int g = find_group(offt, groups, static_cast<uint32_t>(r));
                const int32_t j = ws.ties[static_cast<size_t>(g) * ws.chunk + (r - static_cast<int>(offt[g]))];
                sk[r] = 0u;
                sa[r] = arrival[j];
                si[r] = j;
            } else {
                sk[r] = 0xffffffffu;
                sa[r] = LLONG_MAX;
                si[r] = INT_MAX;
            }
        }
        __syncthreads();
        block_bitonic(sk, sa, si, P);
        for (int r = threadIdx.x; r < static_cast<int>(need0); r += kThreads) ws.picked[r] = si[r];
        npicked = need0;
        __syncthreads();
    } else if (need0 > 0) {
        // Many ties: make the tie list contiguous (in place, moving forward), then a radix
        // selection over the 96-bit (arrival, index) key by this work-group, compacting the
        // list after every digit.
        for (int g = 0; g < groups; ++g) {
            const uint32_t cnt = ws.counts[2 * g + 1];
            // offt[g] <= g * chunk: every sweep reads its sources before any is overwritten.
            for (uint32_t base = 0; base < cnt; base += kThreads) {
                const uint32_t r = base + threadIdx.x;
                int32_t j = 0;
                if (r < cnt) j = ws.ties[static_cast<size_t>(g) * ws.chunk + r];
                __syncthreads();
                if (r < cnt) ws.ties[offt[g] + r] = j;
                __syncthreads();
            }
        }
        uint32_t need = need0;
        int lo = 96;
        while (need > 0 && lo > 0) {
            const int w = lo >= 11 ? 11 : lo;
            lo -= w;
            for (int b = threadIdx.x; b < kBins; b += kThreads) hist[b] = 0u;
            __syncthreads();
            for (uint32_t t = threadIdx.x; t < ntie; t += kThreads) {
                const int32_t j = ws.ties[t];
                atomicAdd(&hist[tie_digit(arrival_key(arrival[j]), static_cast<uint32_t>(j), lo, w)], 1u);
            }
            __syncthreads();
            constexpr int PER = kBins / kThreads;
            uint32_t h[PER], sum = 0;
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                h[q] = hist[threadIdx.x * PER + q];
                sum += h[q];
            }
            scan[threadIdx.x] = sum;
            __syncthreads();
            for (int off = 1; off < kThreads; off <<= 1) {
                const uint32_t v = threadIdx.x >= off ? scan[threadIdx.x - off] : 0u;
                __syncthreads();
                scan[threadIdx.x] += v;
                __syncthreads();
            }
            uint32_t below = scan[threadIdx.x] - sum;
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                if (below < need && need <= below + h[q]) {
                    sh_bucket = threadIdx.x * PER + q;
                    sh_below = below;
                    sh_cnt = h[q];
                }
                below += h[q];
            }
            __syncthreads();
            const uint32_t bucket = sh_bucket;
            const bool take_all = sh_cnt == need - sh_below;
            // digit < bucket (or == bucket when taken whole) -> picked; == bucket -> kept.
            uint32_t kept = 0, picked = npicked;
            for (uint32_t base = 0; base < ntie; base += kThreads) {
                const uint32_t t = base + threadIdx.x;
                int32_t j = 0;
                uint32_t dg = 0xffffffffu;
                if (t < ntie) {
                    j = ws.ties[t];
                    dg = tie_digit(arrival_key(arrival[j]), static_cast<uint32_t>(j), lo, w);
                }
                const bool ch = t < ntie && (dg < bucket || (dg == bucket && take_all));
                const bool kp = t < ntie && dg == bucket && !take_all;
                const uint32_t mine = (ch ? 1u : 0u) | (kp ? 0x10000u : 0u);
                scan[threadIdx.x] = mine;
                __syncthreads();
                for (int off = 1; off < kThreads; off <<= 1) {
                    const uint32_t v = threadIdx.x >= off ? scan[threadIdx.x - off] : 0u;
                    __syncthreads();
                    scan[threadIdx.x] += v;
                    __syncthreads();
                }
                const uint32_t ex = scan[threadIdx.x] - mine, tot = scan[kThreads - 1];
                if (ch) ws.picked[picked + (ex & 0xffffu)] = j;
                if (kp) ws.ties[kept + (ex >> 16)] = j;  // kept + rank <= t: in-place is safe
                picked += tot & 0xffffu;
                kept += tot >> 16;
                __syncthreads();
            }
            need = take_all ? 0u : need - (picked - npicked);
            npicked = picked;
            ntie = kept;
            __syncthreads();
        }
    }
    // The k chosen jobs: nchosen from the scatter plus npicked ties; sort by the full key.
    const int P = pow2_at_least(k);
    for (int r = threadIdx.x; r < P; r += kThreads) {
        if (r < k) {
            int32_t j;
            if (r < static_cast<int>(nchosen)) {
                const int g = find_group(offc, groups, static_cast<uint32_t>(r));
                j = ws.chosen[static_cast<size_t>(g) * kSortMaxN + (r - static_cast<int>(offc[g]))];
            } else {
                j = ws.picked[r - static_cast<int>(nchosen)];
            }
            sk[r] = order_key(pred[j]);
            sa[r] = arrival[j];
            si[r] = j;
        } else {
            sk[r] = 0xffffffffu;
            sa[r] = LLONG_MAX;
            si[r] = INT_MAX;
        }
    }
    __syncthreads();
    block_bitonic(sk, sa, si, P);
    for (int r = threadIdx.x; r < k; r += kThreads) out_idx[r] = si[r];
}

}  // namespace

int select_max_n() { return kLargeMaxN; }
int select_max_k(int n) { return n <= kSortMaxN ? INT_MAX : kSortMaxN; }

namespace {

struct LargePlan {
    int groups, chunk;
};

LargePlan large_plan(int n) {
    // Chunks of at least two sweeps of a 1024-thread work-group reading 4 jobs per thread,
    // a multiple of 4096 jobs (16-byte aligned starts), at most kMaxGroups of them.
    constexpr int kSweep = 4 * kBlock;
    int groups = (n + 2 * kSweep - 1) / (2 * kSweep);
    groups = groups < kMaxGroups ? groups : kMaxGroups;
    const int chunk = ((n + groups - 1) / groups + kSweep - 1) / kSweep * kSweep;
    return LargePlan{(n + chunk - 1) / chunk, chunk};
}

size_t large_layout(int n, LargeWs* ws, char* base) {
    const LargePlan pl = large_plan(n);
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align_up(bytes);
        return base ? base + at : nullptr;
    };
    LargeWs w{};
    w.status = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t)));
    w.state = reinterpret_cast<SelState*>(take(sizeof(SelState)));
    w.totals = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * kBins));
    w.partial = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * kBins * static_cast<size_t>(pl.groups)));
    w.counts = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * 2 * static_cast<size_t>(pl.groups)));
    w.chosen = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * kSortMaxN * static_cast<size_t>(pl.groups)));
    w.ties = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * static_cast<size_t>(n)));
    w.picked = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * kSortMaxN));
    w.chunk = pl.chunk;
    w.groups = pl.groups;
    if (ws) *ws = w;
    return o;
}

}  // namespace

size_t select_workspace_bytes(int n) {
    if (n < 1 || n > kLargeMaxN) return 0;
    if (n <= kSortMaxN) return align_up(sizeof(uint32_t));
    return large_layout(n, nullptr, nullptr);
}

hipError_t launch_select(const float* pred, const int64_t* arrival, int n, int k, int32_t* out_idx,
                         int32_t* out_count, void* workspace, hipStream_t st) {
    if (n < 1 || n > kLargeMaxN || k < 0) return hipErrorInvalidValue;
    uint32_t* status = static_cast<uint32_t*>(workspace);
    if (n <= kRankMaxN) {
        const int threads = (n + kWave - 1) / kWave * kWave;  // one thread per job, whole waves
        ELIS_TRY(launch_kernel(select_rank_kernel, dim3(1), dim3(threads), 0, st, pred, arrival, n, k, out_idx, out_count,
                               status));
        return hipSuccess;
    }
    if (n <= kSortMaxN) {
        ELIS_TRY(launch_kernel(select_sort_kernel, dim3(1), dim3(kThreads), 0, st, pred, arrival, n, k, out_idx, out_count,
                           status));
        return hipSuccess;
    }
    const int kk = k < n ? k : n;
    if (kk > kSortMaxN) return hipErrorInvalidValue;
    LargeWs ws;
    large_layout(n, &ws, static_cast<char*>(workspace));
    ELIS_TRY(launch_kernel(select_init_kernel, dim3(1), dim3(256), 0, st, ws, kk, out_count));
    if (kk == 0) return hipSuccess;
    const dim3 grid(ws.groups), red(kReduceBlocks);
    ELIS_TRY(launch_kernel((select_count_kernel<21, 11>), grid, dim3(kBlock), 0, st, pred, n, ws));
    ELIS_TRY(launch_kernel((select_reduce_kernel<11>), red, dim3(1024), 0, st, ws));
    ELIS_TRY(launch_kernel((select_count_kernel<10, 11>), grid, dim3(kBlock), 0, st, pred, n, ws));
    ELIS_TRY(launch_kernel((select_reduce_kernel<11>), red, dim3(1024), 0, st, ws));
    ELIS_TRY(launch_kernel((select_count_kernel<0, 10>), grid, dim3(kBlock), 0, st, pred, n, ws));
    ELIS_TRY(launch_kernel((select_reduce_kernel<10>), red, dim3(1024), 0, st, ws));
    ELIS_TRY(launch_kernel(select_scatter_kernel, grid, dim3(kBlock), 0, st, pred, n, ws));
    ELIS_TRY(launch_kernel(select_final_kernel, dim3(1), dim3(kThreads), 0, st, pred, arrival, kk, ws, out_idx));
    return hipSuccess;
}

// ---------------------------------------------------------------------------------------------
// Allocation-free select: the same launches as launch_select on a fixed per-device scratch array
// instead of a caller workspace. `scratch` below is a device variable: in host code its name is
// only a stand-in, so the host takes the array's device address once per device with
// hipGetSymbolAddress and passes that address to the kernels. Each launch sequence initialises
// what it reads (select_init_kernel writes the selection state and status; every count, list and
// histogram is stored before it is read), so nothing needs clearing between calls.

namespace {

static_assert(kNoAllocScratchBytes % kAlign == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device, once taken

hipError_t scratch_address(void** out) {
    int dev = 0;
    ELIS_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        ELIS_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

int select_noalloc_max_n() {
    static_assert(kNoAllocMaxN <= kLargeMaxN, "limit");
    return kNoAllocMaxN;
}

hipError_t launch_select_noalloc(const float* pred, const int64_t* arrival, int n, int k, int32_t* out_idx,
                                 int32_t* out_count, hipStream_t st) {
    if (n < 1 || n > kNoAllocMaxN || select_workspace_bytes(n) > kNoAllocScratchBytes) return hipErrorInvalidValue;
    void* ws = nullptr;
    ELIS_TRY(scratch_address(&ws));
    return launch_select(pred, arrival, n, k, out_idx, out_count, ws, st);
}

}  // namespace elis
