// Host-side launchers of the libelis kernels (each defined in its own .hip file).
#pragma once

#include <hip/hip_ext.h>

#include <tuple>

#include "common.h"

namespace elis {

// seqmap.hip: validate cu_seqlens, write the sanitised sequence table and the
// attention tile prefix; overwrites *status with the ELIS_DEV_* bits found.
hipError_t launch_seqmap(const int32_t* cu, int n, int total, int max_seqlen, SeqTable tab,
                         uint32_t* status, hipStream_t st);

// norm.hip
// Row outputs of a LayerNorm y = (z - mean) * rstd * g + b (any pointer may be null):
//   y32   fp32 y;  y16  bf16 y;  z32  the pre-norm row z itself (embedding only);
//   stats (mean, rstd) of the row, from which a later epilogue rebuilds y out of z.
struct LnOut {
    float* y32;
    uint16_t* y16;
    float* z32;
    float2* stats;
};
hipError_t launch_embed_ln(const int32_t* ids, const int32_t* cu, int n, int total,
                           const uint16_t* word, const uint16_t* pos, const float* type0,
                           const float* g, const float* b, int d, int vocab, int max_pos, float eps,
                           LnOut out, uint32_t* status, hipStream_t st);
hipError_t launch_layernorm(const float* x, const float* g, const float* b, int rows, int d, float eps,
                            LnOut out, hipStream_t st);
// dst[s] = src[start[s]] and dst_stats[s] = src_stats[start[s]] for s < n (rows of d floats).
hipError_t launch_gather_rows(const float* src, const float2* src_stats, const int32_t* start, int n, int d,
                              float* dst, float2* dst_stats, hipStream_t st);

// gemm.hip
// Residual added by the fp32-output epilogues: the fp32 matrix x itself (stats null), or the
// LayerNorm output rebuilt from its pre-norm input x: fmaf((x - mean) * rstd, g, b), the same
// expression the LayerNorm kernel evaluates, so both see bit-identical values.
struct Residual {
    const float* x;       // [M, N]
    const float2* stats;  // [M] (mean, rstd), or null
    const float* g;       // [N]
    const float* b;       // [N]
};
// Internal epilogue codes beyond the public ELIS_EPI_*: fp32 output + bias + LayerNorm-form
// residual. Same arithmetic; two instantiations so that the attention output projection and
// the second feed-forward product carry their own kernel names in profiles.
constexpr int kEpiResLn = 4;
constexpr int kEpiResLnFfn2 = 5;

hipError_t launch_gemm(const uint16_t* x, const uint16_t* w, const float* bias, Residual res, int m, int n,
                       int k, int epi, void* out, hipStream_t st);

// Launch plan of one product (gemm.hip): rows [0, m1) with configuration `main`, then, when
// m1 < M, rows [m1, M) with configuration `rest`.
struct GemmPlan {
    int main, m1, rest;
};
GemmPlan plan_gemm(int m, int n, int k, int epi);
hipError_t launch_gemm_plan(const GemmPlan& p, const uint16_t* x, const uint16_t* w, const float* bias,
                            Residual res, int m, int n, int k, int epi, void* out, hipStream_t st);
// Tile of a configuration (zeros if unknown) and the configuration of a tile (-1 if none).
int gemm_config_of_tile(int bm, int bn, int wgs_per_cu);

hipError_t launch_gemm_config(int cfg, int group_m, const uint16_t* x, const uint16_t* w, const float* bias,
                              Residual res, int m, int n, int k, int epi, void* out, hipStream_t st);
void gemm_config_tile(int cfg, int* bm, int* bn, int* wgs_per_cu);

// attention.hip
// cls_only: only the first query of each sequence, written to row s of out ([n, heads * dh]).
hipError_t launch_attention(const uint16_t* qkv, SeqTable tab, int n, int total, int heads, int dh,
                            uint16_t* out, hipStream_t st, bool cls_only = false);

// pool_head.hip
constexpr int kPoolChunk = 64;  // rows per partial sum of mean pooling
struct PoolScratch {
    float* partial;  // [n, nchunk, d]   (mean pooling)
    float* z;        // [n, d]           (mean pooling)
    float* hid;      // [n, head_hidden] (multi-layer head)
    float* hid2;     // [n, head_hidden] (more than two layers: the other ping-pong buffer)
    int nchunk;      // ceil(max_seqlen / kPoolChunk)
};
// The regression head: `layers` FC layers, hidden width `hidden`, activation `act`.
struct HeadSpec {
    int layers, hidden, act;
    const float *w1, *b1, *w2, *b2;
    const float* const* mid_w;  // host array of layers - 2 device pointers
    const float* const* mid_b;
};
hipError_t launch_pool_head(const float* hidden, SeqTable tab, int n, int d, int pooling, const HeadSpec& head,
                            float scale, float shift, float* out, PoolScratch scr, hipStream_t st);

// select.hip
int select_max_n();
int select_max_k(int n);  // largest batch cap accepted for n jobs
size_t select_workspace_bytes(int n);
// workspace: select_workspace_bytes(n) bytes, 256-byte aligned; its first word is the status.
hipError_t launch_select(const float* pred, const int64_t* arrival, int n, int k, int32_t* out_idx,
                         int32_t* out_count, void* workspace, hipStream_t st);
// The same selection on the library's fixed per-device scratch (no workspace, no allocation):
// n <= kNoAllocMaxN jobs; the scratch holds select_workspace_bytes(kNoAllocMaxN).
constexpr int kNoAllocMaxN = ELIS_SELECT_NOALLOC_MAX_N;
constexpr size_t kNoAllocScratchBytes = ELIS_SELECT_NOALLOC_SCRATCH_BYTES;
int select_noalloc_max_n();
hipError_t launch_select_noalloc(const float* pred, const int64_t* arrival, int n, int k, int32_t* out_idx,
                                 int32_t* out_count, hipStream_t st);

// jobs.hip: device-resident job table (first token, ring of the last max_pos - 1 tokens,
// length, cached prediction, arrival) for incremental packing across rounds.
struct JobTable {
    uint32_t* status;
    int32_t* first;    // [J]
    int32_t* len;      // [J]
    float* pred;       // [J]
    int64_t* arrival;  // [J]
    int32_t* ring;     // [J][max_pos - 1]
    int max_jobs, max_pos;
};
size_t jobs_table_bytes(int max_jobs, int max_pos);
JobTable jobs_table(void* base, int max_jobs, int max_pos);
hipError_t launch_jobs_init(JobTable t, hipStream_t st);
hipError_t launch_jobs_start(JobTable t, const int32_t* slots, const int64_t* arrival, int m, hipStream_t st);
hipError_t launch_jobs_append(JobTable t, const int32_t* slots, const int32_t* off, const int32_t* tokens, int m,
                              int total, hipStream_t st);
hipError_t launch_jobs_pack(JobTable t, const int32_t* slots, int n, int total, int max_seqlen, int32_t* ids,
                            int32_t* cu, hipStream_t st);
hipError_t launch_jobs_store_pred(JobTable t, const int32_t* slots, const float* pred, int n, hipStream_t st);
size_t jobs_select_workspace_bytes(int max_active);
// wait: null, or fp32 [a] seconds waited, aging the keys by `aging` tokens per second.
hipError_t launch_jobs_select(JobTable t, const int32_t* slots, const float* wait, float aging, int a, int k,
                              int32_t* out_slots, int32_t* out_count, void* workspace, hipStream_t st);

// ------------------------------------------------------------------ launching
// Timing hook of the opt-in per-class timing (api.hip): while a timed class is
// being enqueued it hands out one start/stop event pair per kernel launch;
// otherwise it returns false and leaves both null.
bool launch_timing_events(hipEvent_t* start, hipEvent_t* stop);

// Returns from the enclosing launcher with the first failing HIP status.
#define ELIS_TRY(expr)                       \
    do {                                     \
        const hipError_t elis_e_ = (expr);   \
        if (elis_e_ != hipSuccess) return elis_e_; \
    } while (0)

// Every kernel of the library is enqueued through launch_kernel. When the hook
// hands out events they travel with the dispatch packet (hipExtLaunchKernel)
// and take its own start and end timestamps, so timing a class puts no marker
// packets, and no extra gaps, between the kernels of a forward pass.
template <typename... P, typename... A>
[[nodiscard]] inline hipError_t launch_kernel(void (*kernel)(P...), dim3 grid, dim3 block, uint32_t lds, hipStream_t st,
                                A... a) {
    static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
    std::tuple<P...> args{static_cast<P>(a)...};
    hipEvent_t start = nullptr, stop = nullptr;
    launch_timing_events(&start, &stop);
    return std::apply(
        [&](auto&... v) {
            void* ptrs[] = {static_cast<void*>(&v)...};
            return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, ptrs, lds, st, start,
                                      stop, 0);
        },
        args);
}

}  // namespace elis
