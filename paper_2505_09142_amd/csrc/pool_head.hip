// Pooling + regression head.
//
// CLS pooling takes the sequence's first final hidden vector (Sec. 3.2); mean
// pooling averages all of them, the CLS position included (Sec. 4.2). The head
// is a stack of fully connected fp32 layers: d->1, or d->hidden, hidden->hidden
// (head_layers - 2 times), hidden->1, with ReLU or no activation between layers
// (the paper's eight-layer, width-1024 head, Sec. 4.2); the result is mapped
// to tokens as shift + scale * y.
//
// Kernels (all reductions in a fixed order, so results are bitwise
// reproducible and independent of how sequences are packed):
//   pool_partial  mean pooling only: per (sequence, 256-column block, 64-row
//                 chunk) column sums, fully coalesced row reads;
//   pool_reduce   mean pooling only: chunk sums in order, divided by the length;
//   head_tile     every layer of a multi-layer head but the last, when the inputs
//                 are a multiple of 64 and the outputs of 16 (every configured
//                 head): one work-group per 16 sequences x 16 output units, its
//                 4 or 8 waves splitting the inputs, each accumulating its part on
//                 the fp32 matrix cores (16 x 16 x 4 blocks); the parts are summed
//                 in a fixed order through LDS. Ping-pongs between two [n, hidden]
//                 buffers;
//   head_fc       the same layer for other widths: one wave per (output unit,
//                 8 sequences), lanes across the inputs;
//   head_out      one wave per sequence: ReLU(hidden + b1) . w2 + b2 (or z . w
//                 + b for the linear head), then shift + scale * y.
// For CLS pooling the head reads the CLS row of the hidden states in place.
#include "kernels.h"

namespace elis {

namespace {

constexpr int kCols = 256;      // columns per pooling work-group
constexpr int kFcSeq = 8;  // sequences sharing one weight-row read in head_fc

template <int ACT>
__device__ __forceinline__ float act(float x) {
    if constexpr (ACT == ELIS_ACT_RELU) return fmaxf(x, 0.f);
    return x;
}

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
    const int m = used < nchunk ? used : nchunk;
    // Chunk sums in chunk order; eight loads in flight per pass.
    constexpr int kU = 8;
    float acc = 0.f;
    for (int c0 = 0; c0 < m; c0 += kU) {
        float v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) v[u] = c0 + u < m ? p[static_cast<size_t>(c0 + u) * d] : 0.f;
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if (c0 + u < m) acc += v[u];
    }
    z[static_cast<size_t>(s) * d + c] = acc / static_cast<float>(L);
}

__device__ __forceinline__ const float* pooled_row(int s, int pooling, const float* hidden, const float* z,
                                                   const int32_t* start, int d) {
    // CLS pooling: the sequence's first row, or row s when the hidden rows are one per sequence
    // (start null: the encoder's last layer ran on the CLS rows only).
    const size_t row = start ? static_cast<size_t>(start[s]) : static_cast<size_t>(s);
    return pooling == ELIS_POOL_CLS ? hidden + row * d : z + static_cast<size_t>(s) * d;
}

// One fully connected layer of the head, out[s, j] = act(x[s, :] . w[j, :] + b[j]), K inputs,
// N outputs: one wave per (output unit, kFcSeq sequences), lanes across K, so a weight row is
// read once per kFcSeq sequences. Many small waves (N * n / kFcSeq) keep load latency hidden;
// the input rows (the pooled rows for the first layer, else the previous layer's output) are
// re-read per unit from L2, which measured cheaper than staging them in LDS for fewer waves.
// grid (N, ceil(n / kFcSeq)), one wave per work-group.
template <int ACT, bool POOLED>
__global__ __launch_bounds__(kWave) void head_fc_kernel(const float* __restrict__ in, const float* __restrict__ hidden,
                                                        const float* __restrict__ z, const int32_t* __restrict__ start,
                                                        int pooling, int n, int K, int N,
                                                        const float* __restrict__ w, const float* __restrict__ b,
                                                        float* __restrict__ out) {
    const int j = blockIdx.x, s0 = blockIdx.y * kFcSeq, lane = threadIdx.x;
    const float* wr = w + static_cast<size_t>(j) * K;
    const float* xr[kFcSeq];
#pragma unroll
    for (int q = 0; q < kFcSeq; ++q) {
        const int s = s0 + q < n ? s0 + q : n - 1;
        xr[q] = POOLED ? pooled_row(s, pooling, hidden, z, start, K) : in + static_cast<size_t>(s) * K;
    }
    float acc[kFcSeq];
#pragma unroll
    for (int q = 0; q < kFcSeq; ++q) acc[q] = 0.f;
    for (int c = 4 * lane; c < K; c += 4 * kWave) {
        const f32x4 wv = *reinterpret_cast<const f32x4*>(wr + c);
#pragma unroll
        for (int q = 0; q < kFcSeq; ++q) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(xr[q] + c);
            acc[q] += (wv[0] * v[0] + wv[1] * v[1]) + (wv[2] * v[2] + wv[3] * v[3]);
        }
    }
#pragma unroll
    for (int q = 0; q < kFcSeq; ++q) {
        const float t = wave_sum(acc[q]);
        if (lane == 0 && s0 + q < n) out[static_cast<size_t>(s0 + q) * N + j] = act<ACT>(t + b[j]);
    }
}

// One fully connected layer, out[s, j] = act(x[s, :] . w[j, :] + b[j]), on the fp32 matrix cores.
// A work-group owns 16 sequences x 16 output units; its NW waves split the K inputs into
// contiguous quarters (eighths). Per 16 inputs a lane loads 4 consecutive inputs of its row and
// of its weight row (16 bytes each) and issues four 16 x 16 x 4 blocks; lane l supplies input
// k0 + 4 (l / 16) + i of row l % 16 to block i, the same k for both operands, so every block
// multiplies matching inputs and the 16 inputs are covered once. A wave's 16 x 16 part sits in
// the accumulator layout (lane l: sequences 4 (l / 16) + {0..3}, unit l % 16); the parts are
// summed through LDS in wave order, the bias added and the activation applied by wave 0.
// Every output depends on its own sequence's row only, in a fixed order: results do not depend
// on how many sequences are batched. grid (N / 16, ceil(n / 16)), NW waves; K % (16 NW) == 0.
template <int ACT, bool POOLED, int NW>
__global__ __launch_bounds__(NW* kWave) void head_tile_kernel(const float* __restrict__ in,
                                                              const float* __restrict__ hidden,
                                                              const float* __restrict__ z,
                                                              const int32_t* __restrict__ start, int pooling, int n,
                                                              int K, int N, const float* __restrict__ w,
                                                              const float* __restrict__ b, float* __restrict__ out) {
    __shared__ f32x4 part[NW][kWave];
    const int o0 = blockIdx.x * 16, s0 = blockIdx.y * 16;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
    const int r = lane & 15, kq = lane >> 4;
    const int s = s0 + r < n ? s0 + r : n - 1;  // rows past the end repeat the last, stored nowhere
    const float* xr = POOLED ? pooled_row(s, pooling, hidden, z, start, K) : in + static_cast<size_t>(s) * K;
    const float* wr = w + static_cast<size_t>(o0 + r) * K;
    // Up to kBatch steps of 16 inputs per pass: all their loads are issued before the first block
    // (a wave's share of K is short, so the pass is bound by one load latency, not by a chain).
    constexpr int kBatch = 8;
    const int kw = K / NW, steps = kw / 16;  // the step count is the same for every lane
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int m0 = 0; m0 < steps; m0 += kBatch) {
        const int k0 = wv * kw + 16 * m0 + 4 * kq;
        f32x4 xv[kBatch], wq[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (m0 + u < steps) {
                xv[u] = *reinterpret_cast<const f32x4*>(xr + k0 + 16 * u);
                wq[u] = *reinterpret_cast<const f32x4*>(wr + k0 + 16 * u);
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (m0 + u < steps) {
#pragma unroll
                for (int i = 0; i < 4; ++i) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[u][i], wq[u][i], acc, 0, 0, 0);
            }
        }
    }
    part[wv][lane] = acc;
    __syncthreads();
    if (wv != 0) return;
    f32x4 t = part[0][lane];
#pragma unroll
    for (int q = 1; q < NW; ++q) t += part[q][lane];
    const int o = o0 + r;
    const float bo = b[o];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int si = s0 + 4 * kq + i;
        if (si < n) out[static_cast<size_t>(si) * N + o] = act<ACT>(t[i] + bo);
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
    // Eight strided elements per lane per pass, all loaded before the first product.
    constexpr int kU = 8;
    float acc = 0.f;
    for (int c0 = lane; c0 < len; c0 += kU * kWave) {
        float xv[kU], wv[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int c = c0 + u * kWave;
            xv[u] = c < len ? x[c] : 0.f;
            wv[u] = c < len ? w2[c] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) acc = fmaf(xv[u], wv[u], acc);
    }
    const float y = wave_sum(acc) + b2[0];
    if (lane == 0) out[s] = shift + scale * y;
}

}  // namespace

namespace {

template <int ACT, bool POOLED>
hipError_t fc(const float* in, const float* hidden, const float* z, const int32_t* start, int pooling, int n, int K,
              int N, const float* w, const float* b, float* out, hipStream_t st) {
    if (N % 16 == 0 && K % 128 == 0) {
        ELIS_TRY(launch_kernel((head_tile_kernel<ACT, POOLED, 8>), dim3(N / 16, (n + 15) / 16), dim3(8 * kWave), 0, st,
                               in, hidden, z, start, pooling, n, K, N, w, b, out));
    } else if (N % 16 == 0 && K % 64 == 0) {
        ELIS_TRY(launch_kernel((head_tile_kernel<ACT, POOLED, 4>), dim3(N / 16, (n + 15) / 16), dim3(4 * kWave), 0, st,
                               in, hidden, z, start, pooling, n, K, N, w, b, out));
    } else {
        ELIS_TRY(launch_kernel((head_fc_kernel<ACT, POOLED>), dim3(N, (n + kFcSeq - 1) / kFcSeq), dim3(kWave), 0, st,
                               in, hidden, z, start, pooling, n, K, N, w, b, out));
    }
    return hipSuccess;
}

hipError_t launch_fc(int act, bool pooled, const float* in, const float* hidden, const float* z,
                     const int32_t* start, int pooling, int n, int K, int N, const float* w, const float* b,
                     float* out, hipStream_t st) {
    if (act == ELIS_ACT_RELU)
        return pooled ? fc<ELIS_ACT_RELU, true>(in, hidden, z, start, pooling, n, K, N, w, b, out, st)
                      : fc<ELIS_ACT_RELU, false>(in, hidden, z, start, pooling, n, K, N, w, b, out, st);
    return pooled ? fc<ELIS_ACT_IDENTITY, true>(in, hidden, z, start, pooling, n, K, N, w, b, out, st)
                  : fc<ELIS_ACT_IDENTITY, false>(in, hidden, z, start, pooling, n, K, N, w, b, out, st);
}

}  // namespace

hipError_t launch_pool_head(const float* hidden, SeqTable tab, int n, int d, int pooling, const HeadSpec& head,
                            float scale, float shift, float* out, PoolScratch scr, hipStream_t st) {
    if (d % 4 != 0) return hipErrorInvalidValue;
    const dim3 cols(n, (d + kCols - 1) / kCols);
    if (pooling == ELIS_POOL_MEAN) {
        ELIS_TRY(launch_kernel(pool_partial_kernel, dim3(n, cols.y, scr.nchunk), dim3(kCols), 0, st, hidden, tab.start,
                           tab.len, d, scr.nchunk, scr.partial));
        ELIS_TRY(launch_kernel(pool_reduce_kernel, cols, dim3(kCols), 0, st, scr.partial, tab.len, d, scr.nchunk, scr.z));
    }
    const int hh = head.layers >= 2 ? head.hidden : 0;
    float* cur = scr.hid;
    if (hh > 0) {
        hipError_t e = launch_fc(head.act, true, nullptr, hidden, scr.z, tab.start, pooling, n, d, hh, head.w1,
                                 head.b1, cur, st);
        if (e != hipSuccess) return e;
        float* nxt = scr.hid2;
        for (int l = 0; l < head.layers - 2; ++l) {
            e = launch_fc(head.act, false, cur, nullptr, nullptr, nullptr, pooling, n, hh, hh, head.mid_w[l],
                          head.mid_b[l], nxt, st);
            if (e != hipSuccess) return e;
            float* t = cur;
            cur = nxt;
            nxt = t;
        }
    }
    ELIS_TRY(launch_kernel(head_out_kernel, dim3(n), dim3(kWave), 0, st, hidden, scr.z, tab.start, d, pooling, hh, cur,
                       head.w2, head.b2, scale, shift, out));
    return hipSuccess;
}

}  // namespace elis
