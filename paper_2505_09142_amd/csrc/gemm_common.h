// Device building blocks of the matrix-core product kernels (gemm.hip): the MFMA
// block types, the XCD-aware work-group remap, direct-to-LDS loads and wait-count helpers.
#pragma once

#include "common.h"

namespace elis {
namespace gemm {

// Work-group id -> tile id. The hardware hands consecutive work-group ids round-robin to the
// 8 XCDs (each with its own L2); the remap gives every XCD one contiguous range of tiles.
__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
    constexpr int kXcd = 8;
    const int per = nblk / kXcd, rem = nblk % kXcd;
    const int xcd = bid % kXcd, local = bid / kXcd;
    return xcd * per + (xcd < rem ? xcd : rem) + local;
}

// One MFMA block of the wave tile: MI x MI outputs (MI = 16: 16x16x32, MI = 32: 32x32x16).
template <int MI>
struct Mfma;

template <>
struct Mfma<16> {
    typedef f32x4 acc_t;
    static constexpr int kRegs = 4;
    static constexpr int kDepth = 32;  // k per instruction
    __device__ static __forceinline__ acc_t run(bf16x8 a, bf16x8 b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

template <>
struct Mfma<32> {
    typedef f32x16 acc_t;
    static constexpr int kRegs = 16;
    static constexpr int kDepth = 16;
    __device__ static __forceinline__ acc_t run(bf16x8 a, bf16x8 b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

typedef __attribute__((address_space(3))) void lds_void_t;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 encoding: vmcnt[3:0] in bits 3:0, vmcnt[5:4] in bits 15:14; expcnt/lgkmcnt left at max.
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// One wave-wide 16-byte-per-lane load from global memory straight into LDS: lane i's 16 bytes
// land at lds + 16 * i.
__device__ __forceinline__ void load_lds_16(const void* src, void* lds) {
    __builtin_amdgcn_global_load_lds(src, (lds_void_t*)lds, 16, 0, 0);
}

__device__ __forceinline__ void block_sync_lds() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int N>
__device__ __forceinline__ void wait_lgkm() {
    __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (N << 8) | (3 << 14));
}

// NM MFMA groups, with NV direct loads and ND LDS reads spread evenly in front of them.
template <int G, int NM, int NV, int ND, int SYNC>
__device__ __forceinline__ void interleave_step() {
    if constexpr (G < NM) {
        constexpr int v = (G + 1) * NV / NM - G * NV / NM;
        constexpr int d = (G + 1) * ND / NM - G * ND / NM;
        if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, SYNC);
        if constexpr (d > 0) __builtin_amdgcn_sched_group_barrier(0x100, d, SYNC);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, SYNC);
        interleave_step<G + 1, NM, NV, ND, SYNC>();
    }
}

}  // namespace gemm
}  // namespace elis
