/*
 * libelis: iterative response-length prediction and ISRTF batch selection
 * on AMD Instinct MI355X (gfx950).
 *
 * ELIS schedules LLM jobs by Iterative Shortest Remaining Time First: at
 * every scheduling iteration each job that just ran (and each new arrival)
 * is re-scored by an encoder-based predictor that reads the prompt followed by
 * the tokens generated so far and outputs the number of tokens the job still
 * has to produce (Sec. 3.3; Alg. 1); the batcher then forms the batch from
 * the jobs with the fewest predicted remaining tokens (Sec. 4.1). The
 * predictor is a BERT-style bidirectional Transformer encoder (BGE, Sec. 3.1)
 * with a pooled regression head (CLS vector: Sec. 3.2; mean pooling: Sec. 4.2).
 *
 * Conventions for every call below:
 *  - All data pointers are DEVICE pointers owned by the caller, unless a
 *    comment says "host". The library allocates no device memory, never frees
 *    caller memory and keeps no state between calls (except the opt-in,
 *    per-thread timing facility at the end of this file, and the fixed
 *    per-device scratch of elis_isrtf_select_noalloc).
 *  - Every call validates its scalar arguments on the host, then only
 *    enqueues kernels on `stream` (a hipStream_t; NULL = the default stream)
 *    and returns. Nothing synchronises except elis_read_status and
 *    elis_timing_read.
 *  - Errors are returned as status codes, never thrown; on an error detected
 *    on the host nothing is enqueued.
 *  - bf16 values are passed as their 16-bit patterns (uint16_t).
 *  - Calls on distinct workspaces may run concurrently; calls that share a
 *    workspace must be ordered by the caller (same stream).
 */
#ifndef ELIS_H
#define ELIS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */
#define ELIS_OK           0
#define ELIS_EINVAL      -1 /* null pointer, count <= 0, batch_cap < 0, bad config            */
#define ELIS_ESHAPE      -2 /* max_seqlen > max_pos or < 1, total_tokens < n_seqs, size limit */
#define ELIS_EWORKSPACE  -3 /* ws_bytes smaller than the matching *_workspace_bytes query      */
#define ELIS_EHIP        -4 /* a HIP launch or runtime call failed                             */
#define ELIS_EDEVICE     -5 /* content error found on the device (see elis_read_status)        */
#define ELIS_EUNSUPPORTED -6 /* a shape this build has no kernel for (see elis_config)          */

/* Device-side content error bits, reported by elis_read_status (ORed). */
#define ELIS_DEV_BAD_TOKEN   1u  /* a token id outside [0, vocab)                    */
#define ELIS_DEV_BAD_CU      2u  /* cu_seqlens[0] != 0, not increasing, or != T at n */
#define ELIS_DEV_LONG_SEQ    4u  /* a sequence longer than max_seqlen               */
#define ELIS_DEV_BAD_SLOT    8u  /* a job-table slot outside [0, max_jobs), or a negative token count */
#define ELIS_DEV_PACK_SIZE  16u  /* packed lengths disagree with the host's total / max, or a job is empty */

/* ------------------------------------------------------------------ model */
#define ELIS_POOL_CLS  0 /* the first token's final hidden vector (Sec. 3.2)              */
#define ELIS_POOL_MEAN 1 /* the mean of all of a sequence's final hidden vectors (Sec. 4.2) */

#define ELIS_ACT_RELU     0 /* ReLU between the head's FC layers (Sec. 4.2)           */
#define ELIS_ACT_IDENTITY 1 /* no activation: a stack of linear layers (Sec. 3.2)     */

/*
 * Encoder shape. Supported by this build: d_model % 64 == 0, d_model <= 2048,
 * d_ff % 64 == 0, d_model / n_heads in {32, 64}, n_layers >= 0; head_layers
 * in [1, 16] with head_hidden == 0 when head_layers == 1 and head_hidden a
 * multiple of 4 in [4, 4096] otherwise. Anything else returns
 * ELIS_EUNSUPPORTED (or ELIS_EINVAL for non-positive sizes).
 *
 * The regression head is head_layers fully connected layers on the pooled
 * vector z: one layer d->1; or d->head_hidden, then head_layers - 2 layers
 * head_hidden->head_hidden, then head_hidden->1, with head_act between
 * consecutive layers (the paper's heads: d->256->ReLU->1 style; eight FC layers
 * of width 1024 with ReLU on mean pooling, Sec. 4.2; eight linear layers on
 * the CLS vector, Sec. 3.2).
 */
typedef struct elis_config {
    int32_t n_layers, d_model, n_heads, d_ff, vocab, max_pos;
    int32_t pooling;      /* ELIS_POOL_CLS or ELIS_POOL_MEAN                        */
    int32_t head_hidden;  /* width of the head's hidden layers (0: one layer d->1)  */
    int32_t head_layers;  /* fully connected layers of the head (>= 1)              */
    int32_t head_act;     /* ELIS_ACT_RELU or ELIS_ACT_IDENTITY                     */
    float ln_eps;         /* LayerNorm epsilon (biased variance)                   */
    float out_scale, out_shift; /* prediction = out_shift + out_scale * head output */
} elis_config;

/* One post-LN encoder layer. Matrices are bf16, row-major [out, in]; the rest fp32. */
typedef struct elis_layer_weights {
    const uint16_t *w_qkv; /* [3d, d]: rows 0..d-1 query, d..2d-1 key, 2d..3d-1 value; head h
                              owns rows h*dh..(h+1)*dh-1 of each block                        */
    const uint16_t *w_o;   /* [d, d]  */
    const uint16_t *w_1;   /* [F, d]  */
    const uint16_t *w_2;   /* [d, F]  */
    const float *b_qkv, *b_o, *b_1, *b_2;      /* [3d], [d], [F], [d] */
    const float *ln1_g, *ln1_b, *ln2_g, *ln2_b; /* [d] each            */
} elis_layer_weights;

typedef struct elis_weights {
    elis_config cfg;
    const uint16_t *word;  /* bf16 [vocab, d]   token embedding                 */
    const uint16_t *pos;   /* bf16 [max_pos, d] learned position embedding      */
    const float *type0;    /* fp32 [d]          token-type-0 row, added to all  */
    const float *emb_ln_g, *emb_ln_b;          /* fp32 [d] embedding LayerNorm  */
    const elis_layer_weights *layers;          /* HOST array of n_layers entries */
    const float *head_w1;  /* fp32 [head_hidden, d]: first layer (head_layers >= 2)   */
    const float *head_b1;  /* fp32 [head_hidden]                                      */
    const float *head_w2;  /* fp32 [1, head_hidden], or [1, d] when head_layers == 1  */
    const float *head_b2;  /* fp32 [1]                                                */
    const float *const *head_mid_w; /* HOST array of head_layers - 2 device pointers,
                                       fp32 [head_hidden, head_hidden] each (NULL if none) */
    const float *const *head_mid_b; /* HOST array of head_layers - 2 device pointers,
                                       fp32 [head_hidden] each                           */
} elis_weights;

/*
 * Bytes of device workspace elis_predict_remaining needs for these sizes
 * (0 when the arguments are invalid). The workspace must be 256-byte aligned.
 */
size_t elis_predict_workspace_bytes(const elis_config *cfg, int32_t total_tokens,
                                    int32_t n_seqs, int32_t max_seqlen);

/*
 * Predicted remaining output tokens of every job of a packed batch
 * (Sec. 3.3: the target after g generated tokens is total minus g; Alg. 1:
 * Predictor.init on the prompt, Predictor.iter on prompt followed by the
 * partial response).
 *
 *  token_ids   int32 [total_tokens]: all sequences back to back, no padding.
 *  cu_seqlens  int32 [n_seqs + 1]: sequence s is token_ids[cu[s] .. cu[s+1]-1];
 *              cu[0] == 0, cu[n_seqs] == total_tokens, every length >= 1 and
 *              <= max_seqlen. Positions restart at 0 for every sequence.
 *  max_seqlen  host int: an upper bound on every length, 1 <= max_seqlen <= max_pos.
 *  out_pred    fp32 [n_seqs]: out_shift + out_scale * head(pool(H_s)).
 *  out_hidden  fp32 [total_tokens, d] final hidden states, or NULL.
 *  workspace   >= elis_predict_workspace_bytes(...) bytes, 256-byte aligned.
 * Content errors in token_ids / cu_seqlens are detected on the device: the
 * kernels clamp every index (no out-of-bounds access), the outputs are then
 * undefined and elis_read_status(workspace) returns ELIS_EDEVICE.
 */
int elis_predict_remaining(const elis_weights *w, const int32_t *token_ids,
                           const int32_t *cu_seqlens, int32_t n_seqs, int32_t total_tokens,
                           int32_t max_seqlen, float *out_pred, float *out_hidden,
                           void *workspace, size_t ws_bytes, void *stream);

/* Largest n accepted by elis_isrtf_select in this build (2^28). */
int32_t elis_select_max_n(void);

/*
 * Largest min(batch_cap, n) accepted for n jobs (0 if n is invalid): unbounded
 * (INT32_MAX) for n <= 8192, where one work-group sorts every job; 8192 above,
 * where the chosen jobs are sorted by one work-group after a device-wide radix
 * selection.
 */
int32_t elis_select_max_batch_cap(int32_t n);

/*
 * Bytes of device workspace elis_isrtf_select needs for n jobs (0 if n is
 * invalid): 256 for n <= 8192, about 4n + 41 KiB above (a tie list of up to n
 * indices plus counters and a 2048-bin histogram).
 */
size_t elis_select_workspace_bytes(int32_t n);

/*
 * ISRTF batch selection (Sec. 4.1, the Batcher of Alg. 1): the indices of the
 * min(batch_cap, n) jobs with the fewest predicted remaining tokens, highest
 * priority first. Ties on the prediction are broken by arrival_seq (earlier
 * first, the FCFS order of Sec. 6.1), then by index. -0 equals +0; NaN (any
 * payload) ranks after +inf, all NaNs equal.
 *
 *  pred        fp32 [n], arrival_seq int64 [n]
 *  out_idx     int32 [batch_cap] (only the first min(batch_cap, n) are written)
 *  out_count   int32 [1] device: set to min(batch_cap, n)
 * batch_cap == 0 is valid (count 0). 1 <= n <= elis_select_max_n() (else
 * ELIS_ESHAPE); min(batch_cap, n) <= elis_select_max_batch_cap(n) (else
 * ELIS_EUNSUPPORTED). Enqueue only; out_idx / out_count are valid once the
 * stream reaches the call.
 */
int elis_isrtf_select(const float *pred, const int64_t *arrival_seq, int32_t n,
                      int32_t batch_cap, int32_t *out_idx, int32_t *out_count,
                      void *workspace, size_t ws_bytes, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): elis_isrtf_select
 * without a workspace argument, the same selection bit for bit. Its scratch is
 * a fixed device array of ELIS_SELECT_NOALLOC_SCRATCH_BYTES inside the library,
 * one per GPU the library runs on, held until the process ends; its device
 * address is looked up on the first call on each device. Nothing is allocated
 * by this call. n <= ELIS_SELECT_NOALLOC_MAX_N (else ELIS_ESHAPE, nothing
 * enqueued); other arguments, limits and errors as elis_isrtf_select. Every
 * call on one GPU shares that GPU's scratch, which keeps what the last call
 * left in it (each call initialises what it reads): calls that can overlap on
 * one GPU (other streams, other host threads) race, and the caller must order
 * them.
 */
#define ELIS_SELECT_NOALLOC_MAX_N (1 << 18)
#define ELIS_SELECT_NOALLOC_SCRATCH_BYTES (3u << 20) /* >= elis_select_workspace_bytes(ELIS_SELECT_NOALLOC_MAX_N) */
int elis_isrtf_select_noalloc(const float *pred, const int64_t *arrival_seq, int32_t n, int32_t batch_cap,
                              int32_t *out_idx, int32_t *out_count, void *stream);

/*
 * Synchronises `stream`, then reads the device error word that the last call
 * on `workspace` left: ELIS_OK, ELIS_EDEVICE, or ELIS_EHIP. When `bits` is not
 * NULL (host pointer) the raw ELIS_DEV_* bits are stored there.
 */
int elis_read_status(const void *workspace, void *stream, uint32_t *bits);

/* Human-readable name of a status code (static string). */
const char *elis_status_string(int status);

/* ------------------------------------------------------------------ device-resident job table
 * The input side of a scheduling round kept in HBM (Alg. 1: the Job Pool is
 * re-predicted from prompt + generated tokens; unchanged jobs keep their
 * prediction). A caller-allocated table of max_jobs slots holds, per job, its
 * first token, a ring of its most recent max_pos - 1 tokens, its length, its
 * last prediction and its arrival sequence number. A round appends only the
 * new tokens, packs the re-score set into token_ids / cu_seqlens on the
 * device (input = the job's tokens, or past max_pos tokens the first one plus
 * the most recent max_pos - 1), stores the new predictions, and selects over
 * the cached predictions of the active jobs. Same conventions as above: plain
 * device pointers, enqueue only, errors returned; content errors (a slot
 * outside [0, max_jobs), packed sizes that disagree with the host's) set
 * ELIS_DEV_* bits in the table's status word (read it with elis_read_status
 * on `base`). A call must not name one slot twice.
 */
typedef struct {
    void *base;       /* device, 256-byte aligned, elis_jobs_table_bytes() bytes */
    int32_t max_jobs; /* slots 0 .. max_jobs-1                                    */
    int32_t max_pos;  /* the encoder's position table (>= 2)                      */
} elis_job_table;

/* Bytes of the table (0 if max_jobs < 1 or max_pos < 2). */
size_t elis_jobs_table_bytes(int32_t max_jobs, int32_t max_pos);

/* Every slot empty (length 0), status cleared. */
int elis_jobs_init(const elis_job_table *t, void *stream);

/* Start jobs: slot[i] becomes empty with arrival_seq[i] (device arrays of m). */
int elis_jobs_start(const elis_job_table *t, const int32_t *slots, const int64_t *arrival_seq, int32_t m,
                    void *stream);

/*
 * Append tokens: job slots[i] (device int32 [m]) gets tokens[tok_offsets[i] ..
 * tok_offsets[i+1]) (device int32 [m+1] offsets, starting at 0; tokens device
 * int32 [total_new], total_new = tok_offsets[m] passed by the host).
 */
int elis_jobs_append(const elis_job_table *t, const int32_t *slots, const int32_t *tok_offsets,
                     const int32_t *tokens, int32_t m, int32_t total_new, void *stream);

/*
 * Pack the predictor input of jobs slots[0..n) back to back: out_token_ids
 * (device int32 [total_tokens]) and out_cu_seqlens (device int32 [n+1]).
 * total_tokens = sum of min(length, max_pos) and max_seqlen (>= every such
 * length, <= max_pos) are host ints the caller keeps from its own bookkeeping;
 * a mismatch sets ELIS_DEV_PACK_SIZE and the output is undefined.
 */
int elis_jobs_pack(const elis_job_table *t, const int32_t *slots, int32_t n, int32_t total_tokens,
                   int32_t max_seqlen, int32_t *out_token_ids, int32_t *out_cu_seqlens, void *stream);

/* Cache predictions: the prediction of job slots[i] becomes pred[i] (device, n). */
int elis_jobs_store_pred(const elis_job_table *t, const int32_t *slots, const float *pred, int32_t n,
                         void *stream);

/* Bytes of workspace elis_jobs_select needs for a active jobs (0 if invalid). */
size_t elis_jobs_select_workspace_bytes(int32_t a);

/*
 * ISRTF select over the cached predictions of the active jobs slots[0..a)
 * (same order and ties as elis_isrtf_select): out_slots (device int32
 * [batch_cap]) gets the chosen job slots, highest priority first, out_count
 * (device int32 [1]) their number. Limits of elis_isrtf_select apply with n = a.
 */
int elis_jobs_select(const elis_job_table *t, const int32_t *slots, int32_t a, int32_t batch_cap,
                     int32_t *out_slots, int32_t *out_count, void *workspace, size_t ws_bytes, void *stream);

/*
 * The same select with aged keys, a starvation control (Sec. 3.4: the
 * frequency of preemption is tunable; the paper gives no formula, this is the
 * library's): candidate i is ranked by
 *     key_i = fl32( fl64(pred[slot_i]) - fl64(aging) * fl64(wait[i]) )
 * evaluated in IEEE fp64 with the product and the difference each rounded
 * (no fused multiply-add) and one final rounding to fp32; ties as
 * elis_isrtf_select. wait (device fp32 [a]) is the time candidate i has
 * waited since it last ran or arrived, in the caller's unit (seconds in the
 * package's loop); aging is the key reduction per unit of waiting (tokens per
 * second), finite (else ELIS_EINVAL). aging = 0 ranks exactly like
 * elis_jobs_select. Other arguments, limits and errors as elis_jobs_select.
 */
int elis_jobs_select_aged(const elis_job_table *t, const int32_t *slots, const float *wait, float aging, int32_t a,
                          int32_t batch_cap, int32_t *out_slots, int32_t *out_count, void *workspace,
                          size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------ building blocks
 * The predictor's kernels, exposed one by one for per-kernel parity tests and
 * measurement. Same conventions as above.
 */

/* Epilogues of elis_linear. */
#define ELIS_EPI_BIAS_BF16      0 /* out bf16 = x W^T + b                        */
#define ELIS_EPI_BIAS_GELU_BF16 1 /* out bf16 = GELU(x W^T + b), erf GELU, 1.5e-6 */
#define ELIS_EPI_BIAS_RES_F32   2 /* out fp32 = x W^T + b + residual             */

/*
 * Dense layer on the matrix cores: out[m, n] = epilogue(sum_k x[m,k] w[n,k] + bias[n]).
 *  x bf16 [m, k] row-major; w bf16 [n, k] row-major ([out, in]); bias fp32 [n];
 *  residual fp32 [m, n] (ELIS_EPI_BIAS_RES_F32 only, else ignored).
 * fp32 accumulation. Requires k % 64 == 0, n % 64 == 0, m >= 1.
 */
int elis_linear(const uint16_t *x, const uint16_t *w, const float *bias, const float *residual,
                int32_t m, int32_t n, int32_t k, int32_t epilogue, void *out, void *stream);

/*
 * How elis_linear (and the encoder's products, whose fp32 epilogue carries the
 * same cost) launches an m x n x k product on the current device. Host only:
 * no GPU work, no synchronisation. out[7] = {main_bm, main_bn, main_wgs, m1,
 * rest_bm, rest_bn, rest_wgs}: rows [0, m1) run in tiles of main_bm x main_bn,
 * main_wgs work-groups per compute unit; when m1 < m, rows [m1, m) run in a
 * second launch in tiles of rest_bm x rest_bn, rest_wgs per compute unit (else
 * the three rest fields are 0). The plan comes from a launch-time model of the
 * tile configurations and the device's compute-unit count; every plan gives
 * bit-identical results (except that the 128 x 64 tile, used only when n is
 * an odd multiple of 64, accumulates with 16 x 16 x 32 blocks). Errors: as
 * elis_linear (ELIS_EINVAL, ELIS_EUNSUPPORTED), and ELIS_EINVAL on a null out.
 */
int elis_linear_plan(int32_t m, int32_t n, int32_t k, int32_t epilogue, int32_t *out);

/*
 * elis_linear with the launch plan given instead of chosen: plan[7] in the
 * layout elis_linear_plan writes. Tiles: 256 x 256 (1 work-group per CU),
 * 128 x 128 (2), 64 x 128 (2 or 1; the latter four-stage), 64 x 64 (4 or 2;
 * the latter four-stage), 128 x 64 (2;
 * single launch, and only for n an odd multiple of 64, where it is the only
 * tile); main_bn and rest_bn must divide n, 1 <= m1 <= m, m1 a multiple of
 * main_bm when m1 < m, rest different from main. Every valid plan gives the
 * same bits as elis_linear; meant for benchmarking and re-fitting the launch
 * model on other hardware. Errors: as elis_linear, and ELIS_EINVAL for a null
 * or invalid plan.
 */
int elis_linear_with_plan(const uint16_t *x, const uint16_t *w, const float *bias, const float *residual,
                          int32_t m, int32_t n, int32_t k, int32_t epilogue, const int32_t *plan, void *out,
                          void *stream);

/* Bytes of workspace elis_attention needs (0 if invalid). */
size_t elis_attention_workspace_bytes(int32_t n_seqs, int32_t total_tokens);

/*
 * Bidirectional multi-head self-attention within each sequence of a packed
 * batch: for every head, softmax(q k^T / sqrt(d_head)) v over the tokens of
 * the same sequence only (an encoder sees its whole input, Sec. 1).
 *  qkv  bf16 [total_tokens, 3 * n_heads * d_head]: per token, the query, key
 *       and value blocks, each head-major (head h at h*d_head).
 *  out  bf16 [total_tokens, n_heads * d_head].
 * d_head in {32, 64}. cu_seqlens as for elis_predict_remaining; content errors
 * set bits readable with elis_read_status(workspace).
 */
int elis_attention(const uint16_t *qkv, const int32_t *cu_seqlens, int32_t n_seqs,
                   int32_t total_tokens, int32_t max_seqlen, int32_t n_heads, int32_t d_head,
                   uint16_t *out, void *workspace, size_t ws_bytes, void *stream);

/*
 * LayerNorm of fp32 rows (biased variance): y = g * (x - mean) / sqrt(var + eps) + b.
 *  x fp32 [rows, d]; out_f32 fp32 [rows, d] or NULL; out_bf16 bf16 [rows, d] or NULL
 *  (at least one output). d % 64 == 0, d <= 2048.
 */
int elis_layernorm(const float *x, const float *g, const float *b, int32_t rows, int32_t d,
                   float eps, float *out_f32, uint16_t *out_bf16, void *stream);

/* Bytes of workspace elis_pool_head needs (0 if the arguments are invalid). */
size_t elis_pool_head_workspace_bytes(const elis_config *cfg, int32_t n_seqs, int32_t max_seqlen);

/*
 * Pooling and regression head alone (the last two steps of
 * elis_predict_remaining): CLS pooling takes each sequence's first row
 * (Sec. 3.2), mean pooling averages all of its rows (Sec. 4.2); then the
 * head's head_layers fully connected layers (Sec. 3.2, Sec. 4.2) and the map
 * to tokens, out_pred[s] = out_shift + out_scale * head(pool(H_s)).
 *  w           only cfg and the head_* fields are read (the encoder pointers may be NULL).
 *  hidden      fp32 [total_tokens, d_model] final hidden states, packed as cu_seqlens says.
 *  cu_seqlens, n_seqs, total_tokens, max_seqlen: as for elis_predict_remaining (content
 *              errors set bits readable with elis_read_status(workspace)).
 *  out_pred    fp32 [n_seqs].
 *  workspace   >= elis_pool_head_workspace_bytes(...) bytes, 256-byte aligned.
 */
int elis_pool_head(const elis_weights *w, const float *hidden, const int32_t *cu_seqlens, int32_t n_seqs,
                   int32_t total_tokens, int32_t max_seqlen, float *out_pred, void *workspace, size_t ws_bytes,
                   void *stream);

/* ------------------------------------------------------------------ timing (opt-in)
 * When a class is enabled, each timed launch of it enqueues its kernels with
 * a start/stop HIP event pair attached to each dispatch (hipExtLaunchKernel),
 * so the events carry the kernels' own start and end times. With a stride s
 * (elis_timing_stride, default 1) only every s-th launch of a class since the
 * last reset is timed; the others run untimed. elis_timing_read synchronises
 * the pending events and returns, per class, the number of timed launches and
 * their summed kernel time (a launch that enqueues several kernels counts
 * once, with the sum of its kernels' times). The state is per host thread:
 * each call acts on the calling thread's own records, and launches made by
 * other threads are not timed. Meant for benchmarks.
 */
#define ELIS_K_SEQMAP    0
#define ELIS_K_EMBED_LN  1
#define ELIS_K_GEMM_QKV  2
#define ELIS_K_ATTENTION 3
#define ELIS_K_GEMM_O    4
#define ELIS_K_LAYERNORM 5
#define ELIS_K_GEMM_FFN1 6
#define ELIS_K_GEMM_FFN2 7
#define ELIS_K_POOL_HEAD 8
#define ELIS_K_SELECT    9
#define ELIS_K_JOBS      10 /* job-table append / pack / store / gather */
#define ELIS_K_COUNT     11

int elis_timing_enable(uint32_t class_mask); /* bit c enables class c; 0 disables */
int elis_timing_stride(int32_t every);       /* every >= 1, else ELIS_EINVAL */
int elis_timing_reset(void);                 /* also restarts the stride count */
int elis_timing_read(int32_t kernel_class, int32_t *launches, double *total_ms);

/* ABI version of this header: 3. */
int32_t elis_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ELIS_H */
