/*
 * bacon.h -- C ABI of the MI355X (gfx950) BACON prefill KV-compression pass.
 *
 * BACON (Boundary Attention CalibratiON) refines the observation-window
 * importance score of a layer's KV cache with last-query evidence and keeps
 * the top-K keys of every KV head.  For each layer l, sequence b and KV head h
 * (paper Sec. 4):
 *
 *   B_i = mean over the W window rows (and the G query heads of the group)
 *         of the causal attention A_{q,i} = softmax_i(q . k_i / sqrt(d))
 *                                      (Sec. 4.1, Eq. window_score; App. A)
 *   Q_i = A_{D,i}, D = last prompt position (Sec. 4.2, Eq. last_query_score)
 *   E   = [Q - B]_+                     (Eq. boundary_residual)
 *   L   = P_r E (truncated box mean)    (Sec. 4.3, Eqs. neighbor_matrix, intra_layer_coherence)
 *   T   = mean of E over the previous min(m, l) layers (Eq. inter_layer_persistence)
 *   V   = E + L + T                     (Eq. structurally_calibrated_evidence)
 *   lambda = gamma Std_M(B) / (Std_M(V) + eps), M = top-min(rho K, |I|) of B over I
 *                                      (Sec. 4.4, Eqs. scale_matching_size/set, lambda_solution)
 *   S   = B + lambda V                  (Eq. bacon_score)
 *   kept = TopK over I of pool_k(S)    (Eq. topk_selection, with the SnapKV pooling;
 *                                      pool_mode picks a variant, see bacon_params)
 *   compacted cache = {K_i, V_i : i kept} followed by the W window rows.
 *
 * Conventions (readings of points the paper leaves open):
 *   - Window rows are the last W prompt positions; the candidate set I is
 *     positions [0, N_b - W); the window itself is always kept.
 *   - GQA: attention is averaged over the G = num_q_heads / num_kv_heads query
 *     heads before E is formed; the budget is per KV head.
 *   - Every top-k orders by score descending, then position ascending.
 *   - Std is the population standard deviation; pooling is a centred average
 *     of odd width over I with the in-range count as divisor.
 *
 * Layouts (all device pointers, row-major, packed without padding):
 *   q_win   [B*W, Hq, d]   last W queries of every sequence (post-RoPE)
 *   k, v    [T, Hkv, d]    T = cu_seqlens[B]
 *   score vectors  [Hkv, T] float32 (B, Q, E, V, S)
 *   lse     [B, Hq, W] float32, natural-log normaliser of each window row
 *   lambda  [B, Hkv] float32
 *   idx     int32; (b, h) owns K_{b,h} entries after those of every earlier
 *           pair in (b, h) order (with one budget per sequence: Hkv*budget_b
 *           entries from Hkv * sum_{b'<b} budget_b', head-major); entries are
 *           positions relative to the sequence start, ascending, and -1 where
 *           the candidate set holds fewer than K_{b,h} positions.
 *   k_out, v_out [sum_b (C_b + W), Hkv, d], C_b = max_h K_{b,h}; for each
 *           (b, h) the rows are the kept rows in ascending position, then the
 *           W window rows, then zero rows up to C_b + W.
 *
 * Element type: BACON_FP32 (float) or BACON_BF16 (bfloat16) for q, k, v and
 * the compacted cache; all scores are float32.  head_dim is 64 or 128.
 *
 * Ownership: the caller owns every device buffer, including the workspace
 * (size from bacon_workspace_bytes, 256-byte aligned), which holds the E
 * history of the current prompt.  The library never allocates device memory;
 * it owns only the host-side context.  One context per stream; a context is
 * not thread-safe.  Device pointers must be 16-byte aligned.
 *
 * Errors: every argument check runs on the host before anything is enqueued;
 * a failing call returns a status, enqueues nothing, and bacon_last_error()
 * gives the reason (per calling thread).  No call synchronises the stream;
 * device faults surface at the caller's next synchronisation.
 */
#ifndef BACON_H
#define BACON_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BACON_OK = 0,
  BACON_ERR_INVALID = 1,      /* bad argument, shape, pointer or batch layout */
  BACON_ERR_UNSUPPORTED = 2,  /* valid but outside what the kernels handle    */
  BACON_ERR_ORDER = 3,        /* layer out of sequence, or no prompt begun    */
  BACON_ERR_WORKSPACE = 4,    /* workspace too small or misaligned            */
  BACON_ERR_HIP = 5           /* a HIP runtime call or kernel launch failed   */
} bacon_status;

typedef enum { BACON_FP32 = 0, BACON_BF16 = 1 } bacon_dtype;

enum { BACON_TERM_E = 1, BACON_TERM_L = 2, BACON_TERM_T = 4 };

/* Method parameters.  Defaults (bacon_default_params): radius 5 and
 * persist_m 4 (Sec. 4.3), rho 2 (Sec. 4.4), gamma 1 and eps 1e-12 (the paper
 * gives no value), pool_kernel 7, use_last_query 1, terms E|L|T,
 * pool_mode BACON_POOL_MEAN_S, head_alloc BACON_ALLOC_GIVEN, alloc_floor 0.2. */
/* Head-wise budgets of the fused calls (App. B: BACON keeps the backbone's
 * allocation and changes only the score within a head).
 *   BACON_ALLOC_GIVEN     the batch's budgets (per sequence or per head).
 *   BACON_ALLOC_ADAPTIVE  AdaKV's allocation of each layer: every KV head
 *                         keeps its top floor(alloc_floor K_b) positions by
 *                         the backbone score (B mean-pooled over the
 *                         candidates with pool_kernel); the sequence's other
 *                         H_kv K_b - H_kv floor(alloc_floor K_b) slots go to
 *                         the highest scores over every head's remaining
 *                         positions (ties: score desc, head asc, position
 *                         asc).  Head h then keeps its K_{b,h} best of S.
 *                         The batch gives budgets per sequence (no
 *                         head_budgets), num_kv_heads <= 32, and the
 *                         compacted cache holds one head per row: sequence
 *                         b's H_kv (K_b + W) rows in head order, head h's
 *                         K_{b,h} kept rows then its W window rows (the same
 *                         bytes as the [rows, Hkv, d] layout).  idx keeps its
 *                         layout with K_{b,h} entries per (b, h). */
typedef enum { BACON_ALLOC_GIVEN = 0, BACON_ALLOC_ADAPTIVE = 1 } bacon_head_alloc;
/* Pooling of the score over the candidate set before the top-K.  The method
 * itself does not pool; the average pool of S is the SnapKV convention it is
 * used with, and the variants serve ablations.  All use a centred window of
 * pool_kernel positions truncated to the candidate set, and every variant
 * keeps the scale-matching set and lambda on the unpooled B.
 *   BACON_POOL_MEAN_S  mean of S = B + lambda V over the window
 *   BACON_POOL_MAX_S   max of S over the window
 *   BACON_POOL_MEAN_B  mean of B over the window, before calibration, plus
 *                      lambda V: pool(B) + lambda V.  In this mode
 *                      bacon_calibrate returns that pooled score on the
 *                      candidates (B + lambda V on the window rows) and
 *                      bacon_select_topk ranks its S without pooling. */
typedef enum { BACON_POOL_MEAN_S = 0, BACON_POOL_MAX_S = 1, BACON_POOL_MEAN_B = 2 } bacon_pool_mode;

typedef struct {
  int32_t radius;          /* r of the coherence neighbourhood, 0..16        */
  int32_t persist_m;       /* m, persistence depth, 0..16                    */
  double rho;              /* scale-matching expansion, > 0; M = floor(rho K)
                              is formed in double (Eq. scale_matching_size) */
  float gamma;             /* calibration strength, >= 0                     */
  float eps;               /* stabiliser in lambda, >= 0                     */
  int32_t pool_kernel;     /* odd width of the average pool of S, 1..33      */
  int32_t use_last_query;  /* 1 = BACON; 0 = window score only (S = B)       */
  uint32_t terms;          /* subset of BACON_TERM_E|L|T included in V       */
  int32_t pool_mode;       /* BACON_POOL_MEAN_S (default), _MAX_S, _MEAN_B   */
  int32_t head_alloc;      /* BACON_ALLOC_GIVEN (default) or _ADAPTIVE       */
  float alloc_floor;       /* alpha of the adaptive allocation, in [0, 1]    */
} bacon_params;

/* Static shape of the model and the largest batch a context will see. */
typedef struct {
  int32_t num_layers;
  int32_t num_q_heads;
  int32_t num_kv_heads;      /* num_q_heads % num_kv_heads == 0              */
  int32_t head_dim;          /* 64 or 128                                    */
  int32_t window;            /* W >= 1, and G*W <= 512                       */
  int32_t max_batch;         /* 1..64                                        */
  int64_t max_total_tokens;  /* upper bound of T                             */
  bacon_dtype dtype;
} bacon_shape;

/* A packed batch.  The arrays live in HOST memory and are copied by the call.
 * cu_seqlens[0] = 0 and W <= N_b = cu_seqlens[b+1]-cu_seqlens[b] <= 131072
 * (bacon_calibrate and bacon_select_topk, whose select holds a sequence in
 * LDS: <= 32768, UNSUPPORTED beyond).
 * Budgets: `head_budgets` [batch][num_kv_heads], when not NULL, gives every
 * (sequence, KV head) its own budget K_{b,h} >= 1 (a head-wise allocation of
 * the backbone method, Sec. 4 Preliminaries, kept as it is); otherwise every
 * KV head of sequence b keeps budgets[b] >= 1 (budgets may be NULL when
 * head_budgets is given). */
typedef struct {
  int32_t batch;
  const int32_t *cu_seqlens;    /* [batch + 1] */
  const int32_t *budgets;       /* [batch], keys kept per KV head, >= 1 */
  const int32_t *head_budgets;  /* optional [batch * num_kv_heads], >= 1 */
} bacon_batch;

typedef struct bacon_ctx bacon_ctx;

/* Fills *p with the defaults listed above. */
void bacon_default_params(bacon_params *p);

/* Bytes of device workspace a context of this shape needs; 0 if the shape or
 * parameters are invalid (see bacon_last_error). */
size_t bacon_workspace_bytes(const bacon_shape *shape, const bacon_params *params);

/* Creates a context over the caller's workspace d_ws (ws_bytes >= the size
 * above, 256-byte aligned).  params may be NULL for the defaults. */
bacon_status bacon_init(bacon_ctx **ctx, const bacon_shape *shape, const bacon_params *params,
                        void *d_ws, size_t ws_bytes);

/* Destroys the host context (the workspace stays the caller's). */
bacon_status bacon_free(bacon_ctx *ctx);

/* Starts a prompt: fixes the sequences (cu_seqlens) used by every layer until
 * the next call and resets the layer counter; the E history starts empty.
 * The budgets of later calls may differ from layer to layer (a per-layer budget
 * schedule: the budget K_{l,h} of the backbone method, Sec. 4 Preliminaries):
 * each call keeps its own
 * batch's budgets and sizes its outputs by them.  Enqueues a small clearing
 * kernel on `stream` (a hipStream_t). */
bacon_status bacon_begin_prompt(bacon_ctx *ctx, const bacon_batch *batch, void *stream);

/* Window score and last-query score of one layer (Eqs. window_score,
 * last_query_score): writes B and Q [Hkv, T] and, if d_lse is not NULL, the
 * window-row normalisers [B, Hq, W].  Reads no history; any layer may be scored. */
bacon_status bacon_score(bacon_ctx *ctx, int32_t layer, const bacon_batch *batch,
                         const void *d_q_win, const void *d_k, float *d_lse,
                         float *d_B, float *d_Q, void *stream);

/* Calibration of one layer (Eqs. boundary_residual .. bacon_score): from B and
 * Q writes S [Hkv, T] and lambda [B, Hkv]; E and V [Hkv, T] when not NULL.
 * Appends E to the prompt's history, so `layer` must be the next layer of the
 * prompt (0, 1, 2, ...) counting calibrate and compress_layer calls. */
bacon_status bacon_calibrate(bacon_ctx *ctx, int32_t layer, const bacon_batch *batch,
                             const float *d_B, const float *d_Q, float *d_S, float *d_lambda,
                             float *d_E, float *d_V, void *stream);

/* Pools S over the candidate set and keeps the top budget_b positions per KV
 * head (Eq. topk_selection); writes idx in the layout above. */
bacon_status bacon_select_topk(bacon_ctx *ctx, const bacon_batch *batch, const float *d_S,
                               int32_t *d_idx, void *stream);

/* Builds the compacted cache from idx (cache construction after Eq.
 * topk_selection); rows are copied bit for bit. */
bacon_status bacon_compact(bacon_ctx *ctx, const bacon_batch *batch, const void *d_k,
                           const void *d_v, const int32_t *d_idx, void *d_k_out,
                           void *d_v_out, void *stream);

/* AdaKV's head-wise allocation of one layer (see BACON_ALLOC_ADAPTIVE) from a
 * window score d_B [Hkv, T] (bacon_score's): writes K_{b,h} to d_budgets
 * [batch, Hkv] (int32, device), for a later call's batch.head_budgets.  Uses
 * the context's pool_kernel and alloc_floor; the batch gives per-sequence
 * budgets.  UNSUPPORTED with more than 32 KV heads. */
bacon_status bacon_allocate_heads(bacon_ctx *ctx, const bacon_batch *batch, const float *d_B,
                                  int32_t *d_budgets, void *stream);

/* Where the fused calls under BACON_ALLOC_ADAPTIVE write each layer's budgets:
 * d_budgets [num_layers, max_batch, Hkv] int32 (device), layer l at offset
 * l * max_batch * Hkv, or NULL to stop.  The caller keeps ownership. */
bacon_status bacon_alloc_output(bacon_ctx *ctx, int32_t *d_budgets);

/* The whole pass for one layer: score, calibrate, select and compact, with the
 * intermediates kept in the workspace.  Same ordering rule as calibrate. */
bacon_status bacon_compress_layer(bacon_ctx *ctx, int32_t layer, const bacon_batch *batch,
                                  const void *d_q_win, const void *d_k, const void *d_v,
                                  int32_t *d_idx, void *d_k_out, void *d_v_out, void *stream);

/* The same pass with the window-row normalisers given by the caller: d_lse
 * [B, Hq, W] float32 holds, for window row w of query head q of sequence b,
 * the natural log of sum_{i <= t_w} exp(q_w . k_i / sqrt(d)) over the row's
 * causal keys (Sec. 4.1; the softmax normaliser that a flash-attention
 * prefill computes for every query row).  The first K pass that forms these
 * normalisers is skipped; with the normalisers of bacon_score the results
 * equal bacon_compress_layer's up to their rounding.  d_lse must be a
 * 4-byte-aligned device pointer (INVALID otherwise); the caller keeps
 * ownership.  Same ordering rule as calibrate. */
bacon_status bacon_compress_layer_lse(bacon_ctx *ctx, int32_t layer, const bacon_batch *batch,
                                      const void *d_q_win, const void *d_k, const void *d_v,
                                      const float *d_lse, int32_t *d_idx, void *d_k_out,
                                      void *d_v_out, void *stream);

/* The whole pass for layers first_layer .. first_layer + num_layers - 1 of a
 * prompt (compression at the end of prefill, when every layer's cache is
 * there): the same results as bacon_compress_layer (or, when d_lse is not
 * NULL, bacon_compress_layer_lse) called for each layer in order, bit for
 * bit.  With every layer's inputs at hand, two layers are in flight: the K
 * pass that forms the next layer's normalisers runs in the launch of this
 * layer's scoring pass, their merge in this layer's calibration launch, and
 * this layer's candidate lists and final top-K and compaction in the next
 * layer's calibration and score launches: three launches per layer, all on
 * `stream`.  A layer's outputs are complete when the call's work on the
 * stream is.  The per-layer arguments are host arrays of num_layers device
 * pointers each, in the layouts of bacon_compress_layer; d_lse is NULL or
 * such an array.  layer_batch is NULL (every layer keeps `batch`'s budgets)
 * or a host array of num_layers batches, one per layer, each with the
 * prompt's cu_seqlens and its own budgets or head_budgets: a per-layer
 * budget schedule K_{l,h} of the backbone method (Sec. 4, Preliminaries);
 * each layer's outputs are sized by its own batch.  first_layer must be the
 * prompt's next layer (ORDER otherwise) and the range must end within
 * num_layers (ORDER).  Every pointer and every layer's batch is checked
 * before the first launch (INVALID if NULL, misaligned, or with other
 * sequences); the caller keeps ownership of all buffers. */
bacon_status bacon_compress_prompt(bacon_ctx *ctx, const bacon_batch *batch, int32_t first_layer,
                                   int32_t num_layers, const void *const *d_q_win,
                                   const void *const *d_k, const void *const *d_v,
                                   const float *const *d_lse, int32_t *const *d_idx,
                                   void *const *d_k_out, void *const *d_v_out,
                                   const bacon_batch *const *layer_batch, void *stream);

/* The window-row normalisers alone (Sec. 4.1): writes d_lse [B, Hq, W]
 * float32 as bacon_compress_layer_lse reads them (natural log of the sum of
 * exp(q_w . k_i / sqrt(d)) over the row's causal keys), from one pass over
 * K.  Reads and writes no history, so it needs no begin_prompt and may run
 * for any layer at any time; it uses the context's normaliser scratch, so
 * calls of one context must not overlap each other (bacon_compress_layer
 * uses the same scratch; bacon_compress_layer_lse does not).  This lets a
 * caller form the normalisers of layer l+1 on a second stream while layer l
 * is selected and compacted.  d_lse must be a 4-byte-aligned device pointer
 * (INVALID otherwise); the caller keeps ownership. */
bacon_status bacon_window_lse(bacon_ctx *ctx, const bacon_batch *batch, const void *d_q_win,
                              const void *d_k, float *d_lse, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * bacon_window_lse without a context or workspace.  Writes d_lse [B, Hq, W]
 * exactly as bacon_window_lse does (the same kernels).  The per-chunk
 * partials and the merged normalisers live in a static device scratch of
 * 4 MiB per GPU, which the library holds from the first call on that GPU
 * until the process ends; a batch whose scratch (num_kv_heads * key chunks
 * * padded window rows * 8 bytes, plus the merged normalisers) exceeds it
 * returns BACON_ERR_WORKSPACE before anything is enqueued.  The call
 * allocates nothing.  Every call on a GPU shares that GPU's scratch: calls
 * that overlap on one GPU (other streams, other threads) race.  shape gives
 * the model (max_batch and max_total_tokens bound the batch as for a
 * context); the method parameters are irrelevant to the normalisers.
 * Pointer and batch checks as for bacon_window_lse. */
bacon_status bacon_window_lse_static(const bacon_shape *shape, const bacon_batch *batch,
                                     const void *d_q_win, const void *d_k, float *d_lse,
                                     void *stream);

/* Test instrumentation of the fused calls (bacon_compress_layer, _lse and
 * bacon_compress_prompt), whose intermediates otherwise stay in the
 * workspace: with all three pointers set, every later layer l of those calls
 * copies, once its lambda is formed,
 *   its window score B           to d_B      + l * Hkv * T   ([Hkv, T] float32),
 *   its evidence V = E + L + T   to d_V      + l * Hkv * T   ([Hkv, T]; valid on
 *                                              the candidate positions only),
 *   lambda                       to d_lambda + l * B * Hkv   ([B, Hkv]),
 * with T the prompt's total tokens and B its batch size; the buffers must hold
 * every layer the calls reach (the caller owns them, 4-byte aligned).  The
 * copies are enqueued on the call's stream between the layer's launches, so
 * the measured schedule itself is unchanged.  All NULL switches it off
 * (the default); a mix of NULL and non-NULL is INVALID. */
bacon_status bacon_debug_capture(bacon_ctx *ctx, float *d_B, float *d_V, float *d_lambda);

/* Test instrumentation: waits for the device, then returns the context's
 * device error word: 0, or 1 if a meeting of the single-read K pass ran out
 * of its bounded wait, or 2 if an adaptive allocation failed its own check
 * (its budgets were then left uniform) (the results of that call are then
 * unspecified; the next bacon_begin_prompt clears the word); -1 if it cannot
 * be read.
 * Synchronises the device, unlike every other call. */
int32_t bacon_debug_device_errors(bacon_ctx *ctx);

/* Sizes of the outputs for a batch: idx entries and compacted rows. */
int64_t bacon_idx_count(const bacon_batch *batch, int32_t num_kv_heads);
int64_t bacon_kept_rows(const bacon_batch *batch, int32_t num_kv_heads, int32_t window);

/* Per-kernel timing with hipEvents around every launch of the context.
 * bacon_profile_read waits for the recorded events, fills up to `max`
 * entries (name, launches, total milliseconds) and returns the count. */
typedef struct {
  char name[32];
  int64_t launches;
  double total_ms;
} bacon_kernel_time;

bacon_status bacon_profile_enable(bacon_ctx *ctx, int32_t enable);
int32_t bacon_profile_read(bacon_ctx *ctx, bacon_kernel_time *out, int32_t max);

const char *bacon_status_string(bacon_status s);
const char *bacon_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* BACON_H */
