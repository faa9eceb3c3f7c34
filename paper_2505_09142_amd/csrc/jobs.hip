// Device-resident job table: the input side of the scheduling round kept in HBM.
//
// Each job's predictor input is its prompt followed by the tokens generated so far
// (Sec. 3.3, Predictor.iter of Alg. 1); past the position table it is the first
// token plus the most recent max_pos - 1 tokens. The table keeps, per job slot:
//   first   the first token
//   ring    the most recent R = max_pos - 1 tokens after the first (position p >= 1
//           of the job's token sequence lives at ring[(p - 1) % R])
//   len     tokens so far (prompt + generated)
//   pred    the last prediction, arrival its arrival sequence number
// so a round appends only the new tokens (at most one window per running job),
// packs the re-score set on the device, stores the new predictions, and selects
// over the cached predictions of every active job. Jobs whose input did not change
// keep their prediction: the encoder is deterministic, so re-scoring them would
// return the same bits (Alg. 1 re-predicts the Job Pool only).
#include "kernels.h"

namespace elis {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool slot_ok(int32_t s, int J) { return s >= 0 && s < J; }

__global__ __launch_bounds__(kThreads) void jobs_init_kernel(JobTable t) {
    const int j = blockIdx.x * kThreads + threadIdx.x;
    if (j == 0) *t.status = 0u;
    if (j < t.max_jobs) {
        t.first[j] = 0;
        t.len[j] = 0;
        t.pred[j] = 0.f;
        t.arrival[j] = 0;
    }
}

__global__ __launch_bounds__(kThreads) void jobs_start_kernel(JobTable t, const int32_t* __restrict__ slots,
                                                              const int64_t* __restrict__ arrival, int m) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= m) return;
    const int32_t s = slots[i];
    if (!slot_ok(s, t.max_jobs)) {
        atomicOr(t.status, ELIS_DEV_BAD_SLOT);
        return;
    }
    t.len[s] = 0;
    t.pred[s] = 0.f;
    t.arrival[s] = arrival[i];
}

// One thread per new token. Of the tokens one call appends to a job, only the first
// token of the job and those among its newest R positions are stored, so no two threads
// write the same ring entry.
__global__ __launch_bounds__(kThreads) void jobs_append_kernel(JobTable t, const int32_t* __restrict__ slots,
                                                               const int32_t* __restrict__ off,
                                                               const int32_t* __restrict__ tokens, int m,
                                                               int total) {
    const int q = blockIdx.x * kThreads + threadIdx.x;
    if (q >= total) return;
    const int e = find_segment(off, m, q);
    const int32_t s = slots[e];
    if (!slot_ok(s, t.max_jobs)) return;  // flagged by jobs_len_kernel
    const int len0 = t.len[s], cnt = off[e + 1] - off[e];
    const int p = len0 + (q - off[e]);
    const int R = t.max_pos - 1;
    if (p == 0) t.first[s] = tokens[q];
    else if (p >= len0 + cnt - R) t.ring[static_cast<size_t>(s) * R + (p - 1) % R] = tokens[q];
}

__global__ __launch_bounds__(kThreads) void jobs_len_kernel(JobTable t, const int32_t* __restrict__ slots,
                                                            const int32_t* __restrict__ off, int m) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= m) return;
    const int32_t s = slots[i];
    const int cnt = off[i + 1] - off[i];
    if (!slot_ok(s, t.max_jobs) || cnt < 0) {
        atomicOr(t.status, ELIS_DEV_BAD_SLOT);
        return;
    }
    t.len[s] += cnt;
}

// One work-group: input lengths min(len, max_pos) of the re-score set, their exclusive
// prefix as cu_seqlens, and a check against the host's total and maximum.
__global__ __launch_bounds__(1024) void jobs_pack_scan_kernel(JobTable t, const int32_t* __restrict__ slots, int n,
                                                              int total, int max_seqlen, int32_t* __restrict__ cu) {
    __shared__ int32_t scan[1024];
    __shared__ int32_t carry_s;
    __shared__ uint32_t bad;
    if (threadIdx.x == 0) {
        carry_s = 0;
        bad = 0u;
        cu[0] = 0;
    }
    __syncthreads();
    for (int base = 0; base < n; base += 1024) {
        const int i = base + threadIdx.x;
        int L = 0;
        if (i < n) {
            const int32_t s = slots[i];
            if (slot_ok(s, t.max_jobs)) {
                L = t.len[s] < t.max_pos ? t.len[s] : t.max_pos;
                if (L > max_seqlen) atomicOr(&bad, ELIS_DEV_PACK_SIZE);
            } else {
                atomicOr(&bad, ELIS_DEV_BAD_SLOT);
            }
            if (L < 1) {  // an empty job cannot be encoded: keep cu increasing, flag it
                atomicOr(&bad, ELIS_DEV_PACK_SIZE);
                L = 1;
            }
        }
        scan[threadIdx.x] = L;
        __syncthreads();
        for (int o = 1; o < 1024; o <<= 1) {
            const int v = threadIdx.x >= o ? scan[threadIdx.x - o] : 0;
            __syncthreads();
            scan[threadIdx.x] += v;
            __syncthreads();
        }
        const int carry = carry_s;
        if (i < n) cu[i + 1] = carry + scan[threadIdx.x];
        __syncthreads();
        if (threadIdx.x == 0) carry_s = carry + scan[1023];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (carry_s != total) bad |= ELIS_DEV_PACK_SIZE;
        if (bad) atomicOr(t.status, bad);
    }
}

// One thread per output token: sequence s by binary search over cu, then the job's token
// at input position i (first token, or ring entry of sequence position p).
__global__ __launch_bounds__(kThreads) void jobs_pack_gather_kernel(JobTable t, const int32_t* __restrict__ slots,
                                                                    int n, int total, const int32_t* __restrict__ cu,
                                                                    int32_t* __restrict__ ids) {
    const int q = blockIdx.x * kThreads + threadIdx.x;
    if (q >= total) return;
    const int sq = find_segment(cu, n, q);
    const int32_t s = slots[sq];
    const int i = q - cu[sq];
    int32_t tok = 0;
    if (slot_ok(s, t.max_jobs) && q < cu[n]) {
        const int len = t.len[s], R = t.max_pos - 1;
        if (i == 0) {
            tok = t.first[s];
        } else if (len >= 1) {
            const int p = len > t.max_pos ? len - R - 1 + i : i;
            tok = t.ring[static_cast<size_t>(s) * R + (p - 1) % R];
        }
    }
    ids[q] = tok;
}

__global__ __launch_bounds__(kThreads) void jobs_store_pred_kernel(JobTable t, const int32_t* __restrict__ slots,
                                                                   const float* __restrict__ pred, int n) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= n) return;
    const int32_t s = slots[i];
    if (!slot_ok(s, t.max_jobs)) {
        atomicOr(t.status, ELIS_DEV_BAD_SLOT);
        return;
    }
    t.pred[s] = pred[i];
}

// Gathers the select keys of the active jobs. With `wait` (seconds each job has waited since
// it last ran, fp32), the key is aged: fl32(key - aging * wait) evaluated in fp64 from the fp32
// operands, with the product and the difference each rounded once (no fused multiply-add), so
// the rank order is reproducible exactly in any IEEE fp64 arithmetic.
__global__ __launch_bounds__(kThreads) void jobs_gather_kernel(JobTable t, const int32_t* __restrict__ slots, int a,
                                                               const float* __restrict__ wait, float aging,
                                                               float* __restrict__ pred, int64_t* __restrict__ arr,
                                                               uint32_t* __restrict__ status) {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i >= a) return;
    const int32_t s = slots[i];
    if (!slot_ok(s, t.max_jobs)) {
        atomicOr(status, ELIS_DEV_BAD_SLOT);
        pred[i] = __int_as_float(0x7fc00000);  // NaN: ranks last
        arr[i] = 0;
        return;
    }
    float key = t.pred[s];
    if (wait) key = __double2float_rn(__dsub_rn(static_cast<double>(key),
                                                __dmul_rn(static_cast<double>(aging), static_cast<double>(wait[i]))));
    pred[i] = key;
    arr[i] = t.arrival[s];
}

// Chosen positions of the active list -> job slots (count read on the device).
__global__ __launch_bounds__(kThreads) void jobs_map_kernel(const int32_t* __restrict__ slots,
                                                            const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ count, int cap,
                                                            int32_t* __restrict__ out) {
    const int r = blockIdx.x * kThreads + threadIdx.x;
    if (r < cap && r < *count) out[r] = slots[idx[r]];
}

dim3 grid_for(long long n) { return dim3(static_cast<unsigned>((n + kThreads - 1) / kThreads)); }

}  // namespace

size_t jobs_table_bytes(int max_jobs, int max_pos) {
    const size_t J = static_cast<size_t>(max_jobs), R = static_cast<size_t>(max_pos - 1);
    return align_up(sizeof(uint32_t)) + align_up(4 * J) + align_up(4 * J) + align_up(4 * J) + align_up(8 * J) +
           align_up(4 * J * R);
}

JobTable jobs_table(void* base, int max_jobs, int max_pos) {
    const size_t J = static_cast<size_t>(max_jobs);
    char* p = static_cast<char*>(base);
    JobTable t;
    size_t o = 0;
    t.status = reinterpret_cast<uint32_t*>(p + o);
    o += align_up(sizeof(uint32_t));
    t.first = reinterpret_cast<int32_t*>(p + o);
    o += align_up(4 * J);
    t.len = reinterpret_cast<int32_t*>(p + o);
    o += align_up(4 * J);
    t.pred = reinterpret_cast<float*>(p + o);
    o += align_up(4 * J);
    t.arrival = reinterpret_cast<int64_t*>(p + o);
    o += align_up(8 * J);
    t.ring = reinterpret_cast<int32_t*>(p + o);
    t.max_jobs = max_jobs;
    t.max_pos = max_pos;
    return t;
}

hipError_t launch_jobs_init(JobTable t, hipStream_t st) {
    ELIS_TRY(launch_kernel(jobs_init_kernel, grid_for(t.max_jobs > 0 ? t.max_jobs : 1), dim3(kThreads), 0, st, t));
    return hipSuccess;
}

hipError_t launch_jobs_start(JobTable t, const int32_t* slots, const int64_t* arrival, int m, hipStream_t st) {
    ELIS_TRY(launch_kernel(jobs_start_kernel, grid_for(m), dim3(kThreads), 0, st, t, slots, arrival, m));
    return hipSuccess;
}

hipError_t launch_jobs_append(JobTable t, const int32_t* slots, const int32_t* off, const int32_t* tokens, int m,
                              int total, hipStream_t st) {
    if (total > 0)
        ELIS_TRY(launch_kernel(jobs_append_kernel, grid_for(total), dim3(kThreads), 0, st, t, slots, off, tokens, m,
                           total));
    ELIS_TRY(launch_kernel(jobs_len_kernel, grid_for(m), dim3(kThreads), 0, st, t, slots, off, m));
    return hipSuccess;
}

hipError_t launch_jobs_pack(JobTable t, const int32_t* slots, int n, int total, int max_seqlen, int32_t* ids,
                            int32_t* cu, hipStream_t st) {
    ELIS_TRY(launch_kernel(jobs_pack_scan_kernel, dim3(1), dim3(1024), 0, st, t, slots, n, total, max_seqlen, cu));
    ELIS_TRY(launch_kernel(jobs_pack_gather_kernel, grid_for(total), dim3(kThreads), 0, st, t, slots, n, total, cu, ids));
    return hipSuccess;
}

hipError_t launch_jobs_store_pred(JobTable t, const int32_t* slots, const float* pred, int n, hipStream_t st) {
    ELIS_TRY(launch_kernel(jobs_store_pred_kernel, grid_for(n), dim3(kThreads), 0, st, t, slots, pred, n));
    return hipSuccess;
}

size_t jobs_select_workspace_bytes(int max_active) {
    const size_t a = static_cast<size_t>(max_active);
    const size_t sel = select_workspace_bytes(max_active);
    if (sel == 0) return 0;
    return align_up(4 * a) + align_up(8 * a) + align_up(4 * a) + sel;
}

hipError_t launch_jobs_select(JobTable t, const int32_t* slots, const float* wait, float aging, int a, int k,
                              int32_t* out_slots, int32_t* out_count, void* workspace, hipStream_t st) {
    const size_t n = static_cast<size_t>(a);
    char* p = static_cast<char*>(workspace);
    float* pred = reinterpret_cast<float*>(p);
    int64_t* arr = reinterpret_cast<int64_t*>(p + align_up(4 * n));
    int32_t* idx = reinterpret_cast<int32_t*>(p + align_up(4 * n) + align_up(8 * n));
    void* sel_ws = p + align_up(4 * n) + align_up(8 * n) + align_up(4 * n);
    // Bad slots are flagged in the table's status word: the select clears its own.
    ELIS_TRY(launch_kernel(jobs_gather_kernel, grid_for(a), dim3(kThreads), 0, st, t, slots, a, wait, aging, pred, arr,
                       t.status));
    hipError_t e = launch_select(pred, arr, a, k, idx, out_count, sel_ws, st);
    if (e != hipSuccess) return e;
    const int kk = k < a ? k : a;
    if (kk > 0) ELIS_TRY(launch_kernel(jobs_map_kernel, grid_for(kk), dim3(kThreads), 0, st, slots, idx, out_count, kk, out_slots));
    return hipSuccess;
}

}  // namespace elis
