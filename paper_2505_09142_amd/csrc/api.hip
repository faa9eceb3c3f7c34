// C ABI of libelis: argument validation, workspace layout and the launch
// sequence of one predictor forward pass. Every call enqueues on the caller's
// stream and returns; no device memory is allocated here.
#include <math.h>
#include <string.h>

#include <vector>

#include "kernels.h"

using namespace elis;

namespace {

// ------------------------------------------------------------------ timing facility
// One record per timed kernel launch; `first` marks the first kernel of a class launch
// (a class launch may enqueue several kernels, e.g. the head's two).
struct TimedLaunch {
    int cls;
    bool first;
    hipEvent_t a, b;
};
// The state belongs to the calling host thread (thread_local): enabling, timed launches,
// reset and read act on that thread's records only, so threads never share it.
struct TimingState {
    uint32_t mask = 0;
    std::vector<TimedLaunch> pending;
    std::vector<hipEvent_t> free_events;
    double ms[ELIS_K_COUNT] = {};
    int32_t count[ELIS_K_COUNT] = {};
    uint32_t stride = 1;             // time one class launch in every `stride`
    uint64_t seen[ELIS_K_COUNT] = {};  // class launches enqueued since the last reset
    int timed_cls = -1;              // class being enqueued under timing, else -1
    bool timed_first = false;
    bool failed = false;
};
thread_local TimingState g_t;

hipEvent_t take_event() {
    if (!g_t.free_events.empty()) {
        hipEvent_t e = g_t.free_events.back();
        g_t.free_events.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Runs one class launch; when its class is being timed, every kernel it enqueues
// carries its own start/stop events (launch_timing_events below).
template <class F>
hipError_t timed(int cls, F&& launch) {
    if (!(g_t.mask & (1u << cls))) return launch();
    if (g_t.seen[cls]++ % g_t.stride != 0) return launch();
    const size_t mark = g_t.pending.size();
    g_t.timed_cls = cls;
    g_t.timed_first = true;
    g_t.failed = false;
    const hipError_t e = launch();
    g_t.timed_cls = -1;
    if (e != hipSuccess) {  // drop the records of a class launch that did not complete
        for (size_t i = mark; i < g_t.pending.size(); ++i) {
            g_t.free_events.push_back(g_t.pending[i].a);
            g_t.free_events.push_back(g_t.pending[i].b);
        }
        g_t.pending.resize(mark);
        return e;
    }
    return g_t.failed ? hipErrorOutOfMemory : hipSuccess;
}

int status_of(hipError_t e) {
    if (e == hipSuccess) return ELIS_OK;
    return e == hipErrorInvalidValue ? ELIS_EINVAL : ELIS_EHIP;
}

// ------------------------------------------------------------------ validation
int check_config(const elis_config* c) {
    if (!c) return ELIS_EINVAL;
    if (c->n_layers < 0 || c->d_model <= 0 || c->n_heads <= 0 || c->d_ff <= 0 || c->vocab <= 0 ||
        c->max_pos <= 0 || c->head_hidden < 0 || c->head_layers < 1)
        return ELIS_EINVAL;
    if (c->head_act != ELIS_ACT_RELU && c->head_act != ELIS_ACT_IDENTITY) return ELIS_EINVAL;
    if ((c->head_layers == 1) != (c->head_hidden == 0)) return ELIS_EINVAL;
    if (c->pooling != ELIS_POOL_CLS && c->pooling != ELIS_POOL_MEAN) return ELIS_EINVAL;
    if (!(c->ln_eps >= 0.f) || !isfinite(c->out_scale) || !isfinite(c->out_shift)) return ELIS_EINVAL;
    if (c->d_model % 64 || c->d_model > 2048 || c->d_ff % 64 || c->d_model % c->n_heads) return ELIS_EUNSUPPORTED;
    const int dh = c->d_model / c->n_heads;
    if (dh != 32 && dh != 64) return ELIS_EUNSUPPORTED;
    if (c->head_hidden > 4096 || c->head_hidden % 4 || c->head_layers > 16) return ELIS_EUNSUPPORTED;
    return ELIS_OK;
}

int check_weights(const elis_weights* w) {
    if (!w) return ELIS_EINVAL;
    int r = check_config(&w->cfg);
    if (r != ELIS_OK) return r;
    if (!w->word || !w->pos || !w->type0 || !w->emb_ln_g || !w->emb_ln_b || !w->head_w2 || !w->head_b2)
        return ELIS_EINVAL;
    if (w->cfg.head_layers >= 2 && (!w->head_w1 || !w->head_b1)) return ELIS_EINVAL;
    if (w->cfg.head_layers > 2) {
        if (!w->head_mid_w || !w->head_mid_b) return ELIS_EINVAL;
        for (int l = 0; l < w->cfg.head_layers - 2; ++l)
            if (!w->head_mid_w[l] || !w->head_mid_b[l]) return ELIS_EINVAL;
    }
    if (w->cfg.n_layers > 0 && !w->layers) return ELIS_EINVAL;
    for (int l = 0; l < w->cfg.n_layers; ++l) {
        const elis_layer_weights& y = w->layers[l];
        if (!y.w_qkv || !y.w_o || !y.w_1 || !y.w_2 || !y.b_qkv || !y.b_o || !y.b_1 || !y.b_2 || !y.ln1_g ||
            !y.ln1_b || !y.ln2_g || !y.ln2_b)
            return ELIS_EINVAL;
    }
    return ELIS_OK;
}

bool aligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) % kAlign) == 0; }

// ------------------------------------------------------------------ workspace layout
struct PredictLayout {
    size_t status, start, len, tile_off, work, x32, xb, qkv, attn, ha, hb, sa, sb, ffn, pool_partial, pool_z,
        head_hid, total;
    int nchunk;
};

PredictLayout predict_layout(const elis_config& c, int T, int n, int max_seqlen) {
    PredictLayout p{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align_up(bytes);
        return at;
    };
    const size_t d = c.d_model, F = c.d_ff, t = T;
    p.status = take(sizeof(uint32_t));
    p.start = take(sizeof(int32_t) * n);
    p.len = take(sizeof(int32_t) * n);
    p.tile_off = take(sizeof(int32_t) * (n + 1));
    if (c.n_layers > 0) p.work = take(4 * sizeof(int32_t) * static_cast<size_t>(attn_work_capacity(n, T)));
    p.x32 = take(4 * t * d);
    if (c.n_layers > 0) {
        p.xb = take(2 * t * d);
        p.qkv = take(2 * t * 3 * d);
        p.attn = take(2 * t * d);
        p.ha = take(4 * t * d);
        p.hb = take(4 * t * d);
        p.sa = take(sizeof(float2) * t);
        p.sb = take(sizeof(float2) * t);
        p.ffn = take(2 * t * F);
    }
    p.nchunk = (max_seqlen + kPoolChunk - 1) / kPoolChunk;
    if (c.pooling == ELIS_POOL_MEAN) {
        p.pool_partial = take(sizeof(float) * static_cast<size_t>(n) * p.nchunk * d);
        p.pool_z = take(sizeof(float) * static_cast<size_t>(n) * d);
    }
    if (c.head_layers >= 2)
        p.head_hid = take(sizeof(float) * static_cast<size_t>(n) * c.head_hidden * (c.head_layers > 2 ? 2 : 1));
    p.total = o;
    return p;
}

int check_head(const elis_weights* w) {
    if (!w) return ELIS_EINVAL;
    int r = check_config(&w->cfg);
    if (r != ELIS_OK) return r;
    if (!w->head_w2 || !w->head_b2) return ELIS_EINVAL;
    if (w->cfg.head_layers >= 2 && (!w->head_w1 || !w->head_b1)) return ELIS_EINVAL;
    if (w->cfg.head_layers > 2) {
        if (!w->head_mid_w || !w->head_mid_b) return ELIS_EINVAL;
        for (int l = 0; l < w->cfg.head_layers - 2; ++l)
            if (!w->head_mid_w[l] || !w->head_mid_b[l]) return ELIS_EINVAL;
    }
    return ELIS_OK;
}

// Workspace of elis_pool_head: status word, sequence table, pooling and head scratch.
struct PoolHeadLayout {
    size_t status, start, len, tile_off, pool_partial, pool_z, head_hid, total;
    int nchunk;
};

PoolHeadLayout pool_head_layout(const elis_config& c, int n, int max_seqlen) {
    PoolHeadLayout p{};
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o += align_up(bytes);
        return at;
    };
    p.status = take(sizeof(uint32_t));
    p.start = take(sizeof(int32_t) * n);
    p.len = take(sizeof(int32_t) * n);
    p.tile_off = take(sizeof(int32_t) * (n + 1));
    p.nchunk = (max_seqlen + kPoolChunk - 1) / kPoolChunk;
    if (c.pooling == ELIS_POOL_MEAN) {
        p.pool_partial = take(sizeof(float) * static_cast<size_t>(n) * p.nchunk * c.d_model);
        p.pool_z = take(sizeof(float) * static_cast<size_t>(n) * c.d_model);
    }
    if (c.head_layers >= 2)
        p.head_hid = take(sizeof(float) * static_cast<size_t>(n) * c.head_hidden * (c.head_layers > 2 ? 2 : 1));
    p.total = o;
    return p;
}

size_t attention_ws(int n, int total) {
    return align_up(sizeof(uint32_t)) + 2 * align_up(sizeof(int32_t) * n) + align_up(sizeof(int32_t) * (n + 1)) +
           align_up(4 * sizeof(int32_t) * static_cast<size_t>(attn_work_capacity(n, total)));
}

template <class T>
T* at(void* base, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

int check_linear(const uint16_t* x, const uint16_t* w, const float* bias, const float* residual, int32_t m,
                 int32_t n, int32_t k, int32_t epilogue, void* out) {
    if (!x || !w || !bias || !out) return ELIS_EINVAL;
    if (epilogue != ELIS_EPI_BIAS_BF16 && epilogue != ELIS_EPI_BIAS_GELU_BF16 && epilogue != ELIS_EPI_BIAS_RES_F32)
        return ELIS_EINVAL;
    if (epilogue == ELIS_EPI_BIAS_RES_F32 && !residual) return ELIS_EINVAL;
    if (m <= 0 || n <= 0 || k <= 0) return ELIS_EINVAL;
    if (n % 64 || k % 64) return ELIS_EUNSUPPORTED;
    return ELIS_OK;
}

int run_linear(const GemmPlan& p, const uint16_t* x, const uint16_t* w, const float* bias, const float* residual,
               int32_t m, int32_t n, int32_t k, int32_t epilogue, void* out, void* stream) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int cls = epilogue == ELIS_EPI_BIAS_GELU_BF16 ? ELIS_K_GEMM_FFN1
                    : epilogue == ELIS_EPI_BIAS_RES_F32 ? ELIS_K_GEMM_FFN2
                                                        : ELIS_K_GEMM_QKV;
    const Residual res{epilogue == ELIS_EPI_BIAS_RES_F32 ? residual : nullptr, nullptr, nullptr, nullptr};
    return status_of(timed(cls, [&] { return launch_gemm_plan(p, x, w, bias, res, m, n, k, epilogue, out, st); }));
}

}  // namespace

bool elis::launch_timing_events(hipEvent_t* start, hipEvent_t* stop) {
    *start = *stop = nullptr;
    if (g_t.timed_cls < 0) return false;
    hipEvent_t a = take_event(), b = take_event();
    if (!a || !b) {
        if (a) g_t.free_events.push_back(a);
        if (b) g_t.free_events.push_back(b);
        g_t.failed = true;
        return false;
    }
    g_t.pending.push_back({g_t.timed_cls, g_t.timed_first, a, b});
    g_t.timed_first = false;
    *start = a;
    *stop = b;
    return true;
}

extern "C" {

int32_t elis_abi_version(void) { return 3; }

const char* elis_status_string(int s) {
    switch (s) {
        case ELIS_OK: return "ELIS_OK";
        case ELIS_EINVAL: return "ELIS_EINVAL: invalid argument";
        case ELIS_ESHAPE: return "ELIS_ESHAPE: inconsistent sizes";
        case ELIS_EWORKSPACE: return "ELIS_EWORKSPACE: workspace too small";
        case ELIS_EHIP: return "ELIS_EHIP: HIP runtime error";
        case ELIS_EDEVICE: return "ELIS_EDEVICE: device-detected content error";
        case ELIS_EUNSUPPORTED: return "ELIS_EUNSUPPORTED: shape not supported by this build";
        default: return "unknown status";
    }
}

size_t elis_predict_workspace_bytes(const elis_config* cfg, int32_t total_tokens, int32_t n_seqs,
                                    int32_t max_seqlen) {
    if (check_config(cfg) != ELIS_OK || n_seqs <= 0 || total_tokens < n_seqs || max_seqlen < 1 ||
        max_seqlen > cfg->max_pos)
        return 0;
    return predict_layout(*cfg, total_tokens, n_seqs, max_seqlen).total;
}

int elis_predict_remaining(const elis_weights* w, const int32_t* token_ids, const int32_t* cu_seqlens,
                           int32_t n_seqs, int32_t total_tokens, int32_t max_seqlen, float* out_pred,
                           float* out_hidden, void* workspace, size_t ws_bytes, void* stream) {
    int r = check_weights(w);
    if (r != ELIS_OK) return r;
    if (!token_ids || !cu_seqlens || !out_pred || !workspace) return ELIS_EINVAL;
    if (n_seqs <= 0 || total_tokens <= 0) return ELIS_EINVAL;
    if (!aligned(workspace)) return ELIS_EINVAL;
    const elis_config& c = w->cfg;
    if (max_seqlen < 1 || max_seqlen > c.max_pos || total_tokens < n_seqs) return ELIS_ESHAPE;
    const PredictLayout p = predict_layout(c, total_tokens, n_seqs, max_seqlen);
    if (ws_bytes < p.total) return ELIS_EWORKSPACE;

    hipStream_t st = static_cast<hipStream_t>(stream);
    const int T = total_tokens, n = n_seqs, d = c.d_model, F = c.d_ff, L = c.n_layers;
    uint32_t* status = at<uint32_t>(workspace, p.status);
    const SeqTable tab{at<int32_t>(workspace, p.start), at<int32_t>(workspace, p.len),
                       at<int32_t>(workspace, p.tile_off), L ? at<int32_t>(workspace, p.work) : nullptr};
    float* x32 = at<float>(workspace, p.x32);
    float* final32 = out_hidden ? out_hidden : x32;
    uint16_t* xb = L ? at<uint16_t>(workspace, p.xb) : nullptr;
    uint16_t* qkv = L ? at<uint16_t>(workspace, p.qkv) : nullptr;
    uint16_t* attn = L ? at<uint16_t>(workspace, p.attn) : nullptr;
    // Pre-norm rows of the two sub-blocks (fp32) and their (mean, rstd): hb/sb hold the
    // embedding sum and then each layer's FFN output, ha/sa the attention sub-block's.
    float* ha = L ? at<float>(workspace, p.ha) : nullptr;
    float* hb = L ? at<float>(workspace, p.hb) : nullptr;
    float2* sa = L ? at<float2>(workspace, p.sa) : nullptr;
    float2* sb = L ? at<float2>(workspace, p.sb) : nullptr;
    uint16_t* ffn = L ? at<uint16_t>(workspace, p.ffn) : nullptr;

    hipError_t e;
    e = timed(ELIS_K_SEQMAP, [&] { return launch_seqmap(cu_seqlens, n, T, max_seqlen, tab, status, st); });
    if (e != hipSuccess) return status_of(e);
    e = timed(ELIS_K_EMBED_LN, [&] {
        const LnOut o = L ? LnOut{nullptr, xb, hb, sb} : LnOut{final32, nullptr, nullptr, nullptr};
        return launch_embed_ln(token_ids, cu_seqlens, n, T, w->word, w->pos, w->type0, w->emb_ln_g, w->emb_ln_b, d,
                               c.vocab, c.max_pos, c.ln_eps, o, status, st);
    });
    if (e != hipSuccess) return status_of(e);
    // LayerNorm parameters of the row held in hb/sb (the input of the next layer).
    const float* prev_g = w->emb_ln_g;
    const float* prev_b = w->emb_ln_b;
    // With CLS pooling and no hidden-state output only the CLS rows of the last layer reach the
    // head: after that layer's QKV product (keys and values of every token), attention, the
    // out-projection, the feed-forward block and both LayerNorms run on the n CLS rows alone.
    // Every kernel computes a row independently of the others (attention a query), so the
    // predictions are bit-identical to the full pass.
    const bool cls_tail = c.pooling == ELIS_POOL_CLS && !out_hidden && L > 0;
    const float* head_in = final32;
    for (int l = 0; l < L; ++l) {
        const elis_layer_weights& y = w->layers[l];
        const bool last = (l == L - 1);
        e = timed(ELIS_K_GEMM_QKV, [&] {
            return launch_gemm(xb, y.w_qkv, y.b_qkv, Residual{}, T, 3 * d, d, ELIS_EPI_BIAS_BF16, qkv, st);
        });
        if (e != hipSuccess) return status_of(e);
        if (last && cls_tail) {
            // One row per sequence, in buffers the full-size layer no longer needs:
            //   attn <- CLS attention rows;  ha/sa <- the residual rows (hb/sb at each start);
            //   x32/sb <- attention sub-block pre-norm rows and stats;  xb, ffn as usual;
            //   ha <- FFN pre-norm rows;  hb <- final hidden rows.
            e = timed(ELIS_K_ATTENTION, [&] {
                return launch_attention(qkv, tab, n, T, c.n_heads, d / c.n_heads, attn, st, true);
            });
            if (e != hipSuccess) return status_of(e);
            e = timed(ELIS_K_GEMM_O, [&] {
                ELIS_TRY(launch_gather_rows(hb, sb, tab.start, n, d, ha, sa, st));
                return launch_gemm(attn, y.w_o, y.b_o, Residual{ha, sa, prev_g, prev_b}, n, d, d, kEpiResLn, x32,
                                   st);
            });
            if (e != hipSuccess) return status_of(e);
            e = timed(ELIS_K_LAYERNORM, [&] {
                return launch_layernorm(x32, y.ln1_g, y.ln1_b, n, d, c.ln_eps, LnOut{nullptr, xb, nullptr, sb}, st);
            });
            if (e != hipSuccess) return status_of(e);
            e = timed(ELIS_K_GEMM_FFN1, [&] {
                return launch_gemm(xb, y.w_1, y.b_1, Residual{}, n, F, d, ELIS_EPI_BIAS_GELU_BF16, ffn, st);
            });
            if (e != hipSuccess) return status_of(e);
            e = timed(ELIS_K_GEMM_FFN2, [&] {
                return launch_gemm(ffn, y.w_2, y.b_2, Residual{x32, sb, y.ln1_g, y.ln1_b}, n, d, F, kEpiResLnFfn2,
                                   ha, st);
            });
            if (e != hipSuccess) return status_of(e);
            e = timed(ELIS_K_LAYERNORM, [&] {
                return launch_layernorm(ha, y.ln2_g, y.ln2_b, n, d, c.ln_eps, LnOut{hb, nullptr, nullptr, nullptr},
                                        st);
            });
            if (e != hipSuccess) return status_of(e);
            head_in = hb;
            break;
        }
        e = timed(ELIS_K_ATTENTION,
                  [&] { return launch_attention(qkv, tab, n, T, c.n_heads, d / c.n_heads, attn, st); });
        if (e != hipSuccess) return status_of(e);
        e = timed(ELIS_K_GEMM_O, [&] {
            return launch_gemm(attn, y.w_o, y.b_o, Residual{hb, sb, prev_g, prev_b}, T, d, d, kEpiResLn, ha, st);
        });
        if (e != hipSuccess) return status_of(e);
        e = timed(ELIS_K_LAYERNORM, [&] {
            return launch_layernorm(ha, y.ln1_g, y.ln1_b, T, d, c.ln_eps, LnOut{nullptr, xb, nullptr, sa}, st);
        });
        if (e != hipSuccess) return status_of(e);
        e = timed(ELIS_K_GEMM_FFN1, [&] {
            return launch_gemm(xb, y.w_1, y.b_1, Residual{}, T, F, d, ELIS_EPI_BIAS_GELU_BF16, ffn, st);
        });
        if (e != hipSuccess) return status_of(e);
        e = timed(ELIS_K_GEMM_FFN2, [&] {
            return launch_gemm(ffn, y.w_2, y.b_2, Residual{ha, sa, y.ln1_g, y.ln1_b}, T, d, F, kEpiResLnFfn2, hb,
                               st);
        });
        if (e != hipSuccess) return status_of(e);
        e = timed(ELIS_K_LAYERNORM, [&] {
            const LnOut o = last ? LnOut{final32, nullptr, nullptr, nullptr} : LnOut{nullptr, xb, nullptr, sb};
            return launch_layernorm(hb, y.ln2_g, y.ln2_b, T, d, c.ln_eps, o, st);
        });
        if (e != hipSuccess) return status_of(e);
        prev_g = y.ln2_g;
        prev_b = y.ln2_b;
    }
    e = timed(ELIS_K_POOL_HEAD, [&] {
        float* hid = c.head_layers >= 2 ? at<float>(workspace, p.head_hid) : nullptr;
        const PoolScratch scr{c.pooling == ELIS_POOL_MEAN ? at<float>(workspace, p.pool_partial) : nullptr,
                              c.pooling == ELIS_POOL_MEAN ? at<float>(workspace, p.pool_z) : nullptr, hid,
                              c.head_layers > 2 ? hid + static_cast<size_t>(n) * c.head_hidden : nullptr, p.nchunk};
        const HeadSpec head{c.head_layers, c.head_hidden, c.head_act, w->head_w1, w->head_b1, w->head_w2,
                            w->head_b2, w->head_mid_w, w->head_mid_b};
        const SeqTable rows{cls_tail ? nullptr : tab.start, tab.len, tab.tile_off};
        return launch_pool_head(head_in, rows, n, d, c.pooling, head, c.out_scale, c.out_shift, out_pred, scr, st);
    });
    return status_of(e);
}

size_t elis_pool_head_workspace_bytes(const elis_config* cfg, int32_t n_seqs, int32_t max_seqlen) {
    if (check_config(cfg) != ELIS_OK || n_seqs <= 0 || max_seqlen < 1 || max_seqlen > cfg->max_pos) return 0;
    return pool_head_layout(*cfg, n_seqs, max_seqlen).total;
}

int elis_pool_head(const elis_weights* w, const float* hidden, const int32_t* cu_seqlens, int32_t n_seqs,
                   int32_t total_tokens, int32_t max_seqlen, float* out_pred, void* workspace, size_t ws_bytes,
                   void* stream) {
    int r = check_head(w);
    if (r != ELIS_OK) return r;
    if (!hidden || !cu_seqlens || !out_pred || !workspace) return ELIS_EINVAL;
    if (n_seqs <= 0 || total_tokens <= 0) return ELIS_EINVAL;
    if (!aligned(workspace)) return ELIS_EINVAL;
    const elis_config& c = w->cfg;
    if (max_seqlen < 1 || max_seqlen > c.max_pos || total_tokens < n_seqs) return ELIS_ESHAPE;
    const PoolHeadLayout p = pool_head_layout(c, n_seqs, max_seqlen);
    if (ws_bytes < p.total) return ELIS_EWORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int n = n_seqs;
    const SeqTable tab{at<int32_t>(workspace, p.start), at<int32_t>(workspace, p.len),
                       at<int32_t>(workspace, p.tile_off)};
    hipError_t e = timed(ELIS_K_SEQMAP, [&] {
        return launch_seqmap(cu_seqlens, n, total_tokens, max_seqlen, tab, at<uint32_t>(workspace, p.status), st);
    });
    if (e != hipSuccess) return status_of(e);
    e = timed(ELIS_K_POOL_HEAD, [&] {
        float* hid = c.head_layers >= 2 ? at<float>(workspace, p.head_hid) : nullptr;
        const PoolScratch scr{c.pooling == ELIS_POOL_MEAN ? at<float>(workspace, p.pool_partial) : nullptr,
                              c.pooling == ELIS_POOL_MEAN ? at<float>(workspace, p.pool_z) : nullptr, hid,
                              c.head_layers > 2 ? hid + static_cast<size_t>(n) * c.head_hidden : nullptr, p.nchunk};
        const HeadSpec head{c.head_layers, c.head_hidden, c.head_act, w->head_w1, w->head_b1, w->head_w2,
                            w->head_b2, w->head_mid_w, w->head_mid_b};
        return launch_pool_head(hidden, tab, n, c.d_model, c.pooling, head, c.out_scale, c.out_shift, out_pred, scr,
                                st);
    });
    return status_of(e);
}

int32_t elis_select_max_n(void) { return select_max_n(); }

int32_t elis_select_max_batch_cap(int32_t n) {
    if (n < 1 || n > select_max_n()) return 0;
    return select_max_k(n);
}

size_t elis_select_workspace_bytes(int32_t n) { return select_workspace_bytes(n); }

int elis_isrtf_select(const float* pred, const int64_t* arrival_seq, int32_t n, int32_t batch_cap,
                      int32_t* out_idx, int32_t* out_count, void* workspace, size_t ws_bytes, void* stream) {
    if (!pred || !arrival_seq || !out_count || !workspace || (batch_cap > 0 && !out_idx)) return ELIS_EINVAL;
    if (n <= 0 || batch_cap < 0) return ELIS_EINVAL;
    if (!aligned(workspace)) return ELIS_EINVAL;
    if (n > select_max_n()) return ELIS_ESHAPE;
    if ((batch_cap < n ? batch_cap : n) > select_max_k(n)) return ELIS_EUNSUPPORTED;
    if (ws_bytes < select_workspace_bytes(n)) return ELIS_EWORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = timed(ELIS_K_SELECT, [&] {
        return launch_select(pred, arrival_seq, n, batch_cap, out_idx, out_count, workspace, st);
    });
    return status_of(e);
}

int elis_isrtf_select_noalloc(const float* pred, const int64_t* arrival_seq, int32_t n, int32_t batch_cap,
                              int32_t* out_idx, int32_t* out_count, void* stream) {
    if (!pred || !arrival_seq || !out_count || (batch_cap > 0 && !out_idx)) return ELIS_EINVAL;
    if (n <= 0 || batch_cap < 0) return ELIS_EINVAL;
    if (n > select_noalloc_max_n()) return ELIS_ESHAPE;
    if ((batch_cap < n ? batch_cap : n) > select_max_k(n)) return ELIS_EUNSUPPORTED;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = timed(ELIS_K_SELECT, [&] {
        return launch_select_noalloc(pred, arrival_seq, n, batch_cap, out_idx, out_count, st);
    });
    return status_of(e);
}

namespace {

int check_table(const elis_job_table* t) {
    if (!t || !t->base || t->max_jobs < 1 || t->max_pos < 2) return ELIS_EINVAL;
    if (!aligned(t->base)) return ELIS_EINVAL;
    return ELIS_OK;
}

}  // namespace

size_t elis_jobs_table_bytes(int32_t max_jobs, int32_t max_pos) {
    if (max_jobs < 1 || max_pos < 2) return 0;
    return jobs_table_bytes(max_jobs, max_pos);
}

int elis_jobs_init(const elis_job_table* t, void* stream) {
    int r = check_table(t);
    if (r != ELIS_OK) return r;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(timed(ELIS_K_JOBS,
                           [&] { return launch_jobs_init(jobs_table(t->base, t->max_jobs, t->max_pos), st); }));
}

int elis_jobs_start(const elis_job_table* t, const int32_t* slots, const int64_t* arrival_seq, int32_t m,
                    void* stream) {
    int r = check_table(t);
    if (r != ELIS_OK) return r;
    if (m < 0 || (m > 0 && (!slots || !arrival_seq))) return ELIS_EINVAL;
    if (m == 0) return ELIS_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(timed(ELIS_K_JOBS, [&] {
        return launch_jobs_start(jobs_table(t->base, t->max_jobs, t->max_pos), slots, arrival_seq, m, st);
    }));
}

int elis_jobs_append(const elis_job_table* t, const int32_t* slots, const int32_t* tok_offsets,
                     const int32_t* tokens, int32_t m, int32_t total_new, void* stream) {
    int r = check_table(t);
    if (r != ELIS_OK) return r;
    if (m < 0 || total_new < 0) return ELIS_EINVAL;
    if (m == 0) return ELIS_OK;
    if (!slots || !tok_offsets || (total_new > 0 && !tokens)) return ELIS_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(timed(ELIS_K_JOBS, [&] {
        return launch_jobs_append(jobs_table(t->base, t->max_jobs, t->max_pos), slots, tok_offsets, tokens, m,
                                  total_new, st);
    }));
}

int elis_jobs_pack(const elis_job_table* t, const int32_t* slots, int32_t n, int32_t total_tokens,
                   int32_t max_seqlen, int32_t* out_token_ids, int32_t* out_cu_seqlens, void* stream) {
    int r = check_table(t);
    if (r != ELIS_OK) return r;
    if (!slots || !out_token_ids || !out_cu_seqlens || n <= 0) return ELIS_EINVAL;
    if (total_tokens < n || max_seqlen < 1 || max_seqlen > t->max_pos) return ELIS_ESHAPE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(timed(ELIS_K_JOBS, [&] {
        return launch_jobs_pack(jobs_table(t->base, t->max_jobs, t->max_pos), slots, n, total_tokens, max_seqlen,
                                out_token_ids, out_cu_seqlens, st);
    }));
}

int elis_jobs_store_pred(const elis_job_table* t, const int32_t* slots, const float* pred, int32_t n,
                         void* stream) {
    int r = check_table(t);
    if (r != ELIS_OK) return r;
    if (n < 0 || (n > 0 && (!slots || !pred))) return ELIS_EINVAL;
    if (n == 0) return ELIS_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(timed(ELIS_K_JOBS, [&] {
        return launch_jobs_store_pred(jobs_table(t->base, t->max_jobs, t->max_pos), slots, pred, n, st);
    }));
}

size_t elis_jobs_select_workspace_bytes(int32_t a) {
    if (a < 1 || a > select_max_n()) return 0;
    return jobs_select_workspace_bytes(a);
}

namespace {

int jobs_select_common(const elis_job_table* t, const int32_t* slots, const float* wait, float aging, int32_t a,
                       int32_t batch_cap, int32_t* out_slots, int32_t* out_count, void* workspace, size_t ws_bytes,
                       void* stream) {
    int r = check_table(t);
    if (r != ELIS_OK) return r;
    if (!slots || !out_count || !workspace || (batch_cap > 0 && !out_slots)) return ELIS_EINVAL;
    if (a <= 0 || batch_cap < 0) return ELIS_EINVAL;
    if (!aligned(workspace)) return ELIS_EINVAL;
    if (a > select_max_n()) return ELIS_ESHAPE;
    if ((batch_cap < a ? batch_cap : a) > select_max_k(a)) return ELIS_EUNSUPPORTED;
    if (ws_bytes < jobs_select_workspace_bytes(a)) return ELIS_EWORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(timed(ELIS_K_SELECT, [&] {
        return launch_jobs_select(jobs_table(t->base, t->max_jobs, t->max_pos), slots, wait, aging, a, batch_cap,
                                  out_slots, out_count, workspace, st);
    }));
}

}  // namespace

int elis_jobs_select(const elis_job_table* t, const int32_t* slots, int32_t a, int32_t batch_cap,
                     int32_t* out_slots, int32_t* out_count, void* workspace, size_t ws_bytes, void* stream) {
    return jobs_select_common(t, slots, nullptr, 0.f, a, batch_cap, out_slots, out_count, workspace, ws_bytes,
                              stream);
}

int elis_jobs_select_aged(const elis_job_table* t, const int32_t* slots, const float* wait, float aging, int32_t a,
                          int32_t batch_cap, int32_t* out_slots, int32_t* out_count, void* workspace,
                          size_t ws_bytes, void* stream) {
    if (!wait || !isfinite(aging)) return ELIS_EINVAL;
    return jobs_select_common(t, slots, wait, aging, a, batch_cap, out_slots, out_count, workspace, ws_bytes,
                              stream);
}

int elis_read_status(const void* workspace, void* stream, uint32_t* bits) {
    if (!workspace) return ELIS_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (hipStreamSynchronize(st) != hipSuccess) return ELIS_EHIP;
    uint32_t v = 0;
    if (hipMemcpy(&v, workspace, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return ELIS_EHIP;
    if (bits) *bits = v;
    return v ? ELIS_EDEVICE : ELIS_OK;
}

int elis_linear(const uint16_t* x, const uint16_t* w, const float* bias, const float* residual, int32_t m, int32_t n,
                int32_t k, int32_t epilogue, void* out, void* stream) {
    const int v = check_linear(x, w, bias, residual, m, n, k, epilogue, out);
    if (v != ELIS_OK) return v;
    return run_linear(plan_gemm(m, n, k, epilogue), x, w, bias, residual, m, n, k, epilogue, out, stream);
}

int elis_linear_with_plan(const uint16_t* x, const uint16_t* w, const float* bias, const float* residual, int32_t m,
                          int32_t n, int32_t k, int32_t epilogue, const int32_t* plan, void* out, void* stream) {
    const int v = check_linear(x, w, bias, residual, m, n, k, epilogue, out);
    if (v != ELIS_OK) return v;
    if (!plan) return ELIS_EINVAL;
    GemmPlan p{gemm_config_of_tile(plan[0], plan[1], plan[2]), plan[3], 0};
    if (p.main < 0 || n % plan[1] != 0 || p.m1 < 1 || p.m1 > m) return ELIS_EINVAL;
    if (p.main == 1 && n % 128 == 0) return ELIS_EINVAL;  // 128 x 64 only where nothing else fits
    if (p.m1 < m) {
        p.rest = gemm_config_of_tile(plan[4], plan[5], plan[6]);
        // the 16 x 16 x 32 configuration accumulates in another order: single launches only
        if (p.rest < 0 || p.rest == p.main || p.main == 1 || p.rest == 1 || n % plan[5] != 0 ||
            p.m1 % plan[0] != 0)
            return ELIS_EINVAL;
    } else if (plan[4] || plan[5] || plan[6]) {
        return ELIS_EINVAL;
    }
    return run_linear(p, x, w, bias, residual, m, n, k, epilogue, out, stream);
}

size_t elis_attention_workspace_bytes(int32_t n_seqs, int32_t total_tokens) {
    if (n_seqs <= 0 || total_tokens < n_seqs) return 0;
    return attention_ws(n_seqs, total_tokens);
}

int elis_attention(const uint16_t* qkv, const int32_t* cu_seqlens, int32_t n_seqs, int32_t total_tokens,
                   int32_t max_seqlen, int32_t n_heads, int32_t d_head, uint16_t* out, void* workspace,
                   size_t ws_bytes, void* stream) {
    if (!qkv || !cu_seqlens || !out || !workspace) return ELIS_EINVAL;
    if (n_seqs <= 0 || total_tokens <= 0 || n_heads <= 0 || d_head <= 0) return ELIS_EINVAL;
    if (!aligned(workspace)) return ELIS_EINVAL;
    if (d_head != 32 && d_head != 64) return ELIS_EUNSUPPORTED;
    if (total_tokens < n_seqs || max_seqlen < 1) return ELIS_ESHAPE;
    if (ws_bytes < attention_ws(n_seqs, total_tokens)) return ELIS_EWORKSPACE;
    hipStream_t st = static_cast<hipStream_t>(stream);
    size_t o = 0;
    uint32_t* status = at<uint32_t>(workspace, o);
    o += align_up(sizeof(uint32_t));
    SeqTable tab;
    tab.start = at<int32_t>(workspace, o);
    o += align_up(sizeof(int32_t) * n_seqs);
    tab.len = at<int32_t>(workspace, o);
    o += align_up(sizeof(int32_t) * n_seqs);
    tab.tile_off = at<int32_t>(workspace, o);
    o += align_up(sizeof(int32_t) * (n_seqs + 1));
    tab.work = at<int32_t>(workspace, o);
    hipError_t e = timed(ELIS_K_SEQMAP,
                         [&] { return launch_seqmap(cu_seqlens, n_seqs, total_tokens, max_seqlen, tab, status, st); });
    if (e != hipSuccess) return status_of(e);
    return status_of(timed(ELIS_K_ATTENTION, [&] {
        return launch_attention(qkv, tab, n_seqs, total_tokens, n_heads, d_head, out, st);
    }));
}

int elis_layernorm(const float* x, const float* g, const float* b, int32_t rows, int32_t d, float eps,
                   float* out_f32, uint16_t* out_bf16, void* stream) {
    if (!x || !g || !b || (!out_f32 && !out_bf16)) return ELIS_EINVAL;
    if (rows <= 0 || d <= 0 || !(eps >= 0.f)) return ELIS_EINVAL;
    if (d % 64 || d > 2048) return ELIS_EUNSUPPORTED;
    hipStream_t st = static_cast<hipStream_t>(stream);
    return status_of(
        timed(ELIS_K_LAYERNORM,
              [&] { return launch_layernorm(x, g, b, rows, d, eps, LnOut{out_f32, out_bf16, nullptr, nullptr}, st); }));
}

int elis_linear_plan(int32_t m, int32_t n, int32_t k, int32_t epilogue, int32_t* out) {
    if (!out || m <= 0 || n <= 0 || k <= 0) return ELIS_EINVAL;
    if (epilogue != ELIS_EPI_BIAS_BF16 && epilogue != ELIS_EPI_BIAS_GELU_BF16 && epilogue != ELIS_EPI_BIAS_RES_F32)
        return ELIS_EINVAL;
    if (n % 64 || k % 64) return ELIS_EUNSUPPORTED;
    const GemmPlan p = plan_gemm(m, n, k, epilogue);
    gemm_config_tile(p.main, &out[0], &out[1], &out[2]);
    out[3] = p.m1;
    out[4] = out[5] = out[6] = 0;
    if (p.m1 < m) gemm_config_tile(p.rest, &out[4], &out[5], &out[6]);
    return ELIS_OK;
}

int elis_timing_enable(uint32_t class_mask) {
    g_t.mask = class_mask & ((1u << ELIS_K_COUNT) - 1);
    return ELIS_OK;
}

int elis_timing_stride(int32_t every) {
    if (every < 1) return ELIS_EINVAL;
    g_t.stride = static_cast<uint32_t>(every);
    return ELIS_OK;
}

int elis_timing_reset(void) {
    for (auto& t : g_t.pending) {
        (void)hipEventSynchronize(t.b);
        g_t.free_events.push_back(t.a);
        g_t.free_events.push_back(t.b);
    }
    g_t.pending.clear();
    for (int i = 0; i < ELIS_K_COUNT; ++i) {
        g_t.ms[i] = 0.0;
        g_t.count[i] = 0;
        g_t.seen[i] = 0;
    }
    return ELIS_OK;
}

int elis_timing_read(int32_t kernel_class, int32_t* launches, double* total_ms) {
    if (kernel_class < 0 || kernel_class >= ELIS_K_COUNT || !launches || !total_ms) return ELIS_EINVAL;
    for (auto& t : g_t.pending) {
        if (hipEventSynchronize(t.b) != hipSuccess) return ELIS_EHIP;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, t.a, t.b) != hipSuccess) return ELIS_EHIP;
        g_t.ms[t.cls] += ms;
        g_t.count[t.cls] += t.first ? 1 : 0;
        g_t.free_events.push_back(t.a);
        g_t.free_events.push_back(t.b);
    }
    g_t.pending.clear();
    *launches = g_t.count[kernel_class];
    *total_ms = g_t.ms[kernel_class];
    return ELIS_OK;
}

}  // extern "C"
