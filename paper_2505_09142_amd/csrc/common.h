// Shared device helpers for the libelis kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "elis.h"

namespace elis {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16 bit pattern, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    __bf16 h = static_cast<__bf16>(f);
    return __builtin_bit_cast(uint16_t, h);
}

// Two fp32 -> packed pair of bf16 (lo in the low half), round to nearest even: one
// v_cvt_pk_bf16_f32 (converting the halves separately and merging them costs four instructions).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2 v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

// Largest s in [0, n) with cu[s] <= t, for a non-decreasing cu (clamped for any cu).
__device__ __forceinline__ int find_segment(const int32_t* cu, int n, int t) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (cu[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return lo;
}

}  // namespace elis

// --------------------------------------------------------------------------- host side
// Workspace layout of elis_predict_remaining / elis_attention (all offsets 256-aligned).
namespace elis {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Sequence table written by the seq-map kernel: sanitised start/length of
// every sequence, the exclusive prefix of attention query tiles and, when work
// is not null, the attention work list: one entry {start, length, first query,
// sequence} per query tile, longest sequences first.
struct SeqTable {
    int32_t* start;     // [n]
    int32_t* len;       // [n]
    int32_t* tile_off;  // [n + 1]
    int32_t* work = nullptr;  // [4 * attn_work_capacity(n, total)]
};

// Rows per attention work-group (query tile) used to build the tile table.
constexpr int kAttnRowsPerBlock = 128;

// Entries of the attention work list: sum_s ceil(len_s / 128) <= total / 128 + n for
// lengths that partition the batch; entries past it (malformed lengths) are dropped.
inline int attn_work_capacity(int n, int total) { return (total + kAttnRowsPerBlock - 1) / kAttnRowsPerBlock + n; }

}  // namespace elis
