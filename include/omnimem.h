/*
 * omnimem.h -- C ABI of the OmniMem per-chunk KV-cache compression step on
 * AMD Instinct MI355X (gfx950).
 *
 * Method: OmniMem, "Perturbation-aware Memory Compression for Streaming
 * Audio-Visual LLMs" (arXiv 2606.07577), Sec. 3.  After a chunk has been
 * prefilled, each layer's working set is its retained visual and audio
 * caches followed by the chunk's new KV pairs (Eq. 3).  The step
 *
 *   1. scores every working-set row by accumulated chunk attention (Eq. 6),
 *   2. scores its redundancy by value-vector cosine similarity (Eq. 7),
 *   3. derives per-layer and per-modality budgets from normalised attention
 *      entropy and mean cosine (AVBA, Eqs. 9-14),
 *   4. keeps the top-M rows per modality by psi = a^lambda (1 - s) (Eq. 8,
 *      Eqs. 4-5) and compacts them into the next caches (Eq. 2).
 *
 * The four calls below are those four stages.  They are independent: a
 * caller may supply its own a, s or budgets to any later stage.
 *
 * Conventions shared by every call
 *  - All tensor pointers are DEVICE pointers owned by the caller, except the
 *    `layers` descriptor array, which is a HOST array of cfg.n_layers
 *    entries that is copied before the call returns.
 *  - Every call validates its arguments on the host first; on failure it
 *    returns a nonzero status, launches nothing and sets the text that
 *    omnimem_last_error() returns.
 *  - Work is enqueued asynchronously on `stream`; outputs are valid once the
 *    stream has reached the call's end.  Calls on one context must not run
 *    concurrently (one context per stream).
 *  - No call allocates device memory after omnimem_create().
 *  - Working-set layout of layer l, KV head g (Eq. 3): row j of k, v at
 *    k + g*kv_head_stride + j*kv_row_stride (elements), head_dim contiguous
 *    elements per row.  Rows 0 .. n_cache-1 are the retained caches, rows
 *    n_cache .. n_cache+n_chunk-1 the chunk in time order.  modality[j] is 0
 *    (visual) or 1 (audio) for every row.
 *  - Query head h reads KV head h / (n_q_heads / n_kv_heads) (grouped-query
 *    attention).  Chunk query i of head h is at q + h*q_head_stride +
 *    i*q_row_stride.
 *  - Per-token outputs a, s and idx are [n_layers][n_kv_heads][max_tokens]
 *    row-major; entries past layer l's N = n_cache + n_chunk are untouched.
 *  - Scores, statistics and log-sum-exp values are always fp32.
 */
#ifndef OMNIMEM_H
#define OMNIMEM_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OMNIMEM_OK = 0,
  OMNIMEM_ERR_INVALID_ARG = 1,  /* null pointer, bad size, bad stride, overlap  */
  OMNIMEM_ERR_UNSUPPORTED = 2,  /* head_dim other than 64 or 128, dtype, ...    */
  OMNIMEM_ERR_INFEASIBLE = 3,   /* per-layer minimum budgets exceed the total   */
  OMNIMEM_ERR_CAPACITY = 4,     /* sizes beyond those given to omnimem_create   */
  OMNIMEM_ERR_HIP = 5           /* a HIP runtime error (text in last_error)     */
} omnimem_status;

typedef enum { OMNIMEM_BF16 = 0, OMNIMEM_F32 = 1 } omnimem_dtype;

/* Redundancy source of Eq. (7).  SIM_MAX: s_k = max cosine between row k
 * and any other row of the same (layer, KV head, modality).  SIM_ADJ: the
 * mean cosine with the previous and next row of the same modality (Eq. 7
 * as printed; one neighbour at either end, 0 for a lone row). */
typedef enum { OMNIMEM_SIM_MAX = 0, OMNIMEM_SIM_ADJ = 1 } omnimem_sim;

/* Vectors the cosines of Eq. (7) are taken on.  Eq. (7) is printed on the
 * hidden states; Sec. 3.1 allows the value vectors instead, which keeps the
 * cache as it is.  Hidden states are per token, so one redundancy serves
 * every KV head of the layer; both SIM_ADJ and SIM_MAX apply to them
 * (SIM_MAX with hidden_dim a multiple of 64). */
typedef enum { OMNIMEM_SRC_VALUES = 0, OMNIMEM_SRC_KEYS = 1, OMNIMEM_SRC_HIDDEN = 2 } omnimem_source;

typedef struct {
  int32_t n_layers;      /* L                                                 */
  int32_t n_q_heads;     /* H_q                                               */
  int32_t n_kv_heads;    /* H_kv; must divide H_q                              */
  int32_t head_dim;      /* d: 64 or 128                                       */
  int32_t dtype;         /* omnimem_dtype of q, k, v, k_out, v_out             */
  float lambda;          /* Eq. (8) exponent; paper default 0.02 (Sec. 4.3)    */
  float ratio_r;         /* Eqs. (11)-(12) prior visual:audio ratio; 5         */
  float temperature;     /* Eq. (14) T; 0.2                                    */
  float b_min_frac;      /* per-layer budget >= ceil(b_min_frac*B_tot/L)       */
  float b_max_frac;      /* per-layer budget <= floor(b_max_frac*B_tot/L)      */
  int32_t causal;        /* 1: chunk row n_cache+t is visible to query i iff t <= i */
  int32_t sim;           /* omnimem_sim                                        */
  int32_t sim_source;    /* omnimem_source                                     */
  int32_t shared_selection; /* 0: kept rows per KV head; 1: one set per layer
                             (Eqs. 4-5 carry no head index), ranked by a
                             summed and s averaged over the KV heads      */
  int64_t max_tokens;    /* capacity: largest N = n_cache + n_chunk of a layer */
  int64_t max_chunk;     /* capacity: largest n_chunk of a layer               */
  int32_t hidden_dim;    /* d_model of the hidden states (SRC_HIDDEN); rows of
                            whole 16-byte units                               */
  int32_t inplace_stage_rows; /* in-place compaction (k_out == k): rows per
                            (layer, KV head) reserved for kept rows that land
                            behind their working-set row (audio rows behind a
                            visual block that grew); 0: outputs may not alias
                            the inputs.  See omnimem_select_compact.         */
} omnimem_config;

typedef struct {
  const void* q;            /* [H_q][n_chunk][d] chunk queries                */
  int64_t q_head_stride;    /* elements between query heads                   */
  int64_t q_row_stride;     /* elements between chunk queries                 */
  const void* k;            /* [H_kv][N][d] working-set keys (Eq. 3)           */
  const void* v;            /* [H_kv][N][d] working-set values                 */
  int64_t kv_head_stride;   /* elements, shared by k and v                    */
  int64_t kv_row_stride;    /* elements, shared by k and v; with bf16, below
                               2^24 bytes and times max_tokens below 2^31
                               bytes (rows are addressed by 32-bit byte
                               offsets from a head's base)                  */
  const uint8_t* modality;  /* [N]: 0 visual, 1 audio                         */
  int64_t n_cache;          /* retained rows at the front of the working set  */
  int64_t n_chunk;          /* chunk rows (and chunk queries) at the back     */
  float sm_scale;           /* softmax scale of Eq. (1); 0 -> 1/sqrt(d)        */
  const float* lse;         /* optional [H_q][n_chunk] fp32 log-sum-exp of the
                               chunk attention rows (e.g. from the prefill);
                               NULL -> computed by omnimem_score               */
  void* k_out;              /* [H_kv][M_l][d] next keys   (select_compact)    */
  void* v_out;              /* [H_kv][M_l][d] next values (select_compact)    */
  int64_t out_head_stride;  /* elements, shared by k_out and v_out            */
  int64_t out_row_stride;   /* elements, shared by k_out and v_out            */
  const void* hidden;       /* [N][hidden_dim] hidden states of the working-set
                               rows (SRC_HIDDEN), cfg.dtype                   */
  int64_t hidden_row_stride;   /* elements                                   */
  void* hidden_out;         /* optional [M_l][hidden_dim] hidden states of the
                               kept rows (select_compact, shared selection)   */
  int64_t hidden_out_row_stride; /* elements                                 */
  int64_t out_rows;         /* rows per KV head that k_out / v_out hold;
                               0 -> N (select_compact)                        */
  uint8_t* modality_out;    /* optional [out_rows] modality of the kept rows
                               (select_compact); may equal `modality`         */
} omnimem_layer;

/* One layer's new chunk (Eq. 3): its K and V rows [H_kv][n_rows][d] and the
 * modality of each row, in time order (input of omnimem_append). */
typedef struct {
  const void* k;
  const void* v;
  int64_t head_stride;      /* elements, shared by k and v                    */
  int64_t row_stride;       /* elements, shared by k and v                    */
  const uint8_t* modality;  /* [n_rows]: 0 visual, 1 audio                     */
  int64_t n_rows;           /* must equal the layer descriptor's n_chunk      */
} omnimem_chunk;

typedef struct omnimem_ctx omnimem_ctx;

/* Fill *cfg with the paper's defaults (lambda 0.02, r 5, T 0.2; Sec. 3.2 and
 * Sec. 4.3), b_min_frac 0.5, b_max_frac 2, causal, SIM_MAX on values, bf16.
 * Sizes are left 0. */
void omnimem_config_default(omnimem_config* cfg);

/* Create a context on the current HIP device.  Allocates every workspace
 * buffer for cfg's capacities.  On success *out owns them until
 * omnimem_destroy.  Errors: INVALID_ARG (null, nonpositive sizes, H_kv not
 * dividing H_q), UNSUPPORTED (head_dim, dtype), HIP (allocation failed). */
omnimem_status omnimem_create(const omnimem_config* cfg, omnimem_ctx** out);

/* Wait for the context's outstanding work, free its workspace and the
 * context.  NULL is accepted. */
omnimem_status omnimem_destroy(omnimem_ctx* ctx);

/* Text of the last error on this context ("" if none).  Valid until the next
 * call on the context.  ctx NULL -> text of the last failed omnimem_create. */
const char* omnimem_last_error(const omnimem_ctx* ctx);

/* Eq. (6): a[l][g][j] = sum over query heads h of KV head g and chunk queries
 * i of A_{h,i,j}, A the softmax over visible rows of sm_scale <q_{h,i}, k_{g,j}>
 * (Eq. 1: one softmax over both caches and the chunk).  Each layer's lse is
 * taken from the descriptor when given, else computed.
 *   a       [L][H_kv][max_tokens] fp32, written for j < N_l.
 *   lse_out optional [L][H_q][max_chunk] fp32: the log-sum-exp per chunk query
 *           that was used (copied from the descriptor when given).  */
omnimem_status omnimem_score(omnimem_ctx* ctx, const omnimem_layer* layers, float* a,
                             float* lse_out, hipStream_t stream);

/* Eq. (7): s[l][g][j] = redundancy of row j among the rows of its modality
 * in KV head g, from cfg.sim and cfg.sim_source (with SRC_HIDDEN the one
 * value of each token, from its hidden state, in every head's row).
 * Cosine similarity is 0
 * when either vector is zero and is clamped to [-1, 1]; a modality with a
 * single row gives s = 0.
 *   s [L][H_kv][max_tokens] fp32, written for j < N_l. */
omnimem_status omnimem_redundancy(omnimem_ctx* ctx, const omnimem_layer* layers, float* s,
                                  hipStream_t stream);

/* AVBA, Eqs. (9)-(14): per layer, normalised attention entropy per KV head
 * (averaged over heads) and mean redundancy over visual rows, audio rows and
 * all rows give C_v, C_a (Eqs. 9-10) and C^(l) (Eq. 13, normalised by ln N).
 * Layer shares x_l = clamp(kappa*B_tot*softmax(C/T)_l, lo_l, hi_l) with the
 * kappa making sum x_l = B_tot, lo_l = min(ceil(b_min_frac*B_tot/L), N_l),
 * hi_l = min(floor(b_max_frac*B_tot/L), N_l) (every layer keeps hi_l when
 * sum hi_l <= B_tot).  Integer B_l by largest remainder (ties to the lower
 * layer).  M_v = clamp(floor(w_v*B_l + 1/2), max(0, B_l - K_a), min(K_v, B_l))
 * with w_v from Eq. (11), M_a = B_l - M_v.  Computed in fp64 on the device.
 *   a, s     [L][H_kv][max_tokens] fp32 inputs.
 *   budgets  [L][2] int32 output (M_v, M_a).
 *   stats    optional [L][10] fp32 output: Hn_v, Hn_a, Hn_l, sbar_v, sbar_a,
 *            sbar_l, C_v, C_a, C_l, w_v.
 * Errors: INFEASIBLE when sum_l lo_l > total_budget (checked on the host). */
omnimem_status omnimem_allocate(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a,
                                const float* s, int64_t total_budget, int32_t* budgets,
                                float* stats, hipStream_t stream);

/* omnimem_allocate for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): no context, and no device allocation by this call or by the
 * library on its behalf.  Same arguments and results as omnimem_allocate,
 * with the configuration passed directly (its sizes and options checked as
 * by omnimem_create).  Its scratch (the layer table and the per-chunk
 * partial sums) is a fixed 4 MiB device array of the library, one per GPU,
 * held until the process ends; the call needs under 256 bytes per layer
 * for the table plus L * H_kv * ceil(max_tokens / 512) * 64 bytes of
 * partial sums, and fails with OMNIMEM_ERR_CAPACITY beyond 4 MiB, before
 * any launch (the 28-layer, 4-KV-head, 10240-token stream needs 150 KB).  Every call on a GPU
 * uses the same array: calls that overlap in time on one GPU (on different
 * streams, or from different threads) race and must not be made.  Errors
 * and their text as omnimem_allocate (text from omnimem_last_error(NULL)). */
omnimem_status omnimem_allocate_noalloc(const omnimem_config* cfg, const omnimem_layer* layers, const float* a,
                                        const float* s, int64_t total_budget, int32_t* budgets, float* stats,
                                        hipStream_t stream);

/* Offline budgets (end of Sec. 3.2: the layer budgets may be fixed ahead of
 * time from a few calibration chunks).  The per-layer budgets B^(l) of Eq. (14)
 * are fixed in advance; every step then only splits them between the
 * modalities (Eqs. 11-12).
 *
 * omnimem_calibrate: adds each layer's C^(l) (Eq. 13) of one step, from a
 * and s laid out as for omnimem_allocate, to the context's calibration sums
 * (the first step after create or a reset starts them).  stats, if not
 * null, receives the step's [L][10] statistics as omnimem_allocate writes
 * them.  The sums live in the context's device workspace: calls on one
 * context must be ordered on one stream. */
omnimem_status omnimem_calibrate(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a,
                                 const float* s, float* stats, hipStream_t stream);

/* Forget the calibration steps added so far (host-side: no device work). */
omnimem_status omnimem_calibration_reset(omnimem_ctx* ctx);

/* Layer budgets of the calibration: with C^(l) the mean over the steps added
 * since the last reset, x_l and the integer B_l as in omnimem_allocate, but
 * with lo = ceil(b_min_frac*B_tot/L) and hi = floor(b_max_frac*B_tot/L) for
 * every layer (no token count caps them).  Sum B_l = total_budget unless
 * L*hi < total_budget, when every layer gets hi.
 *   layer_budgets  [L] int32 device output.
 * Errors: INVALID_ARG when no step was added or total_budget is outside
 * [0, 2^31); INFEASIBLE when L*lo > total_budget (checked on the host). */
omnimem_status omnimem_calibration_budgets(omnimem_ctx* ctx, int64_t total_budget,
                                           int32_t* layer_budgets, hipStream_t stream);

/* One step under offline budgets: B_l = min(max(layer_budgets[l], 0), N_l),
 * then M_v, M_a as in omnimem_allocate from this step's w_v (Eq. 11).
 *   a, s           [L][H_kv][max_tokens] fp32 inputs.
 *   layer_budgets  [L] int32 device input (omnimem_calibration_budgets
 *                  writes one).
 *   budgets        [L][2] int32 output (M_v, M_a); stats as above. */
omnimem_status omnimem_allocate_fixed(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a,
                                      const float* s, const int32_t* layer_budgets, int32_t* budgets,
                                      float* stats, hipStream_t stream);

/* Eqs. (4)-(5), (8): per (layer, KV head, modality) keep the M rows with the
 * largest psi = a^lambda (1 - s) (0^lambda = 0; ties to the lower row), in
 * ascending row order, visual block first; then k_out[g][i] = k[g][idx[g][i]]
 * and the same for v, for i < M_v + M_a.  The next step's modality mask is
 * M_v zeros followed by M_a ones.  With cfg.shared_selection the kept rows
 * are chosen once per (layer, modality), by psi of the summed a and the mean
 * s over the layer's KV heads (summed in head order, fp32), and every head
 * keeps them: the idx rows of a layer are then identical, and a layer whose
 * hidden_out is given also gets hidden_out[i] = hidden[idx[l][0][i]]
 * (INVALID_ARG without shared selection or with hidden_out overlapping
 * hidden).
 *   a, s     [L][H_kv][max_tokens] fp32; budgets [L][2] int32 (device).
 *   idx      optional [L][H_kv][max_tokens] int32 output of the kept rows.
 * Budgets are read on the device and applied as M_v = min(max(budget_v, 0),
 * K_v, out_rows) and M_a = min(max(budget_a, 0), K_a, out_rows - M_v): rows
 * beyond a layer's output capacity are not kept, audio rows first.  A layer
 * whose modality_out is given gets modality_out[i] = 0 for i < M_v and 1
 * for M_v <= i < M_v + M_a (it may be the layer's own modality array).
 *
 * Outputs and inputs: k_out / v_out either do not overlap k, v or each
 * other (out of place: the caller ping-pongs two caches), or they ARE k and
 * v (same pointers and strides: in place, as the paper prunes each cache
 * into its next self, Eqs. 2-5); any other overlap is INVALID_ARG.  In place
 * needs cfg.inplace_stage_rows > 0 and gives bit for bit the out-of-place
 * result.  Kept visual rows and most kept audio rows move toward the front
 * and are moved in one ordered pass; kept audio rows that land behind their
 * own row (when M_v exceeds the visual rows in front of them) are first
 * copied to the context's staging rows.  If some (layer, KV head) needs more
 * staging rows than cfg.inplace_stage_rows, the call moves no row of any
 * layer (k, v and modality_out stay as they were; idx is written) and
 * records the shortfall for omnimem_inplace_status.  The hidden states are
 * never compacted in place: hidden_out must not overlap hidden. */
omnimem_status omnimem_select_compact(omnimem_ctx* ctx, const omnimem_layer* layers,
                                      const float* a, const float* s, const int32_t* budgets,
                                      int32_t* idx, hipStream_t stream);

/* Status of the in-place compactions since the last query: OMNIMEM_OK, or
 * OMNIMEM_ERR_CAPACITY when one of them needed more staging rows than the
 * context reserves and so moved nothing (*rows_needed, if not null, gets
 * the largest need; 0 when none), or OMNIMEM_ERR_HIP if an ordering wait of
 * the in-place pass gave up (it waits only on work that has started, so
 * this is not expected).  Synchronous: waits for the device, reads the
 * context's record and clears it. */
omnimem_status omnimem_inplace_status(omnimem_ctx* ctx, int64_t* rows_needed);

/* Eq. (3): each layer's working set is its retained caches followed by the
 * new chunk.  Copies chunks[l]'s K and V rows and modality to rows
 * n_cache .. n_cache + n_chunk - 1 of layers[l].k, .v and .modality (the
 * working-set buffers, written here: the caller owns them and they must be
 * writable), for every layer, in one launch.  The retained rows 0 ..
 * n_cache - 1 are not touched (after an in-place omnimem_select_compact
 * with modality_out = modality they already hold the kept rows and their
 * modality).  This is the write the model's prefill makes when it appends
 * the chunk's K/V behind the cache.
 * Errors: INVALID_ARG (null pointers, alignment, strides, n_rows differing
 * from n_chunk, chunk rows overlapping the destination rows). */
omnimem_status omnimem_append(omnimem_ctx* ctx, const omnimem_layer* layers, const omnimem_chunk* chunks,
                              hipStream_t stream);

/* How omnimem_select_compact ranks the rows (Eq. 8 keys, top M per
 * modality).  Every path keeps the same rows (the top M by psi, ties to the
 * lower row); they differ in speed only.
 *   REGISTERS     one workgroup per (layer, KV head, modality) holding every
 *                 key in registers; working sets of at most 8192 rows.
 *   ONE_WORKGROUP one workgroup per (layer, KV head, modality), keys in LDS
 *                 (in global memory past 32768 rows of a modality).
 *   SPLIT         several workgroups per (layer, KV head) in 2048-row
 *                 slices, three launches: keys and a global first-digit
 *                 histogram, the threshold bin's keys listed, then ranked
 *                 exactly and the rows emitted; at most 524288 rows.
 *   AUTO          REGISTERS up to 8192 rows, ONE_WORKGROUP up to 16384,
 *                 SPLIT beyond (by the call's longest working set).
 * A call whose sizes a chosen path cannot take uses ONE_WORKGROUP.  The
 * setting applies to later calls on the context.
 * Errors: INVALID_ARG (null context, unknown path). */
typedef enum {
  OMNIMEM_TOPK_AUTO = 0,
  OMNIMEM_TOPK_REGISTERS = 1,
  OMNIMEM_TOPK_ONE_WORKGROUP = 2,
  OMNIMEM_TOPK_SPLIT = 3
} omnimem_topk_path;
omnimem_status omnimem_set_topk_path(omnimem_ctx* ctx, int32_t path);

/* Kernel timing for measurement.  While on, every kernel the context
 * launches is bracketed by two HIP events recorded on its launch stream
 * (up to 16384 launches are kept; later ones are not recorded). */
omnimem_status omnimem_profile(omnimem_ctx* ctx, int32_t on);

typedef struct {
  char name[32];       /* kernel name                                       */
  int32_t launches;    /* recorded launches                                 */
  double total_ms;     /* summed event-to-event time of those launches      */
} omnimem_kernel_time;

/* Wait for the recorded launches, write up to `capacity` per-kernel totals
 * (in first-launch order) and their number to *count, and clear the record. */
omnimem_status omnimem_profile_report(omnimem_ctx* ctx, omnimem_kernel_time* out, int32_t capacity,
                                      int32_t* count);

#ifdef __cplusplus
}
#endif

#endif /* OMNIMEM_H */
