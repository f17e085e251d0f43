/*
 * bacon_ref.h -- fp64 CPU oracle of the BACON prefill KV-compression pass.
 *
 * TEST INFRASTRUCTURE ONLY.  This oracle exists to check the HIP path; only
 * the tests, the smoke check and the benchmark's CPU-baseline leg may load it.
 * It shares no code with the GPU library and must never be used as a
 * fallback for it.
 *
 * Method (paper Sec. 4): per layer l, sequence b and KV head h,
 *   window score  B_i = mean over window rows of causal attention A_{q,i}
 *                  (Sec. 4.1, Eq. window_score; softmax scale 1/sqrt(d), App. A)
 *   last query    Q_i = A_{D,i}, D the last prompt position (Eq. last_query_score)
 *   residual      E = [Q - B]_+                     (Eq. boundary_residual)
 *   coherence     L = P_r E, truncated box filter   (Eq. neighbor_matrix, intra_layer_coherence)
 *   persistence   T = mean of E over up to m earlier layers (Eq. inter_layer_persistence)
 *   evidence      V = E + L + T                     (Eq. structurally_calibrated_evidence)
 *   scale         lambda = gamma Std_M(B) / (Std_M(V) + eps),  M = top-rho*K of B
 *                                                   (Sec. 4.4, Eqs. scale_matching_*, lambda_solution)
 *   score         S = B + lambda V                  (Eq. bacon_score)
 *   selection     top-K over the candidate set      (Eq. topk_selection), after an
 *                 average pool of S (the SnapKV pooling convention), or one of
 *                 the pooling variants of pool_mode
 *   cache         keep {K_i, V_i : i selected} plus the window rows.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - GQA: attention is averaged over the G query heads of a KV head before E.
 *   - Window W = last W prompt positions; B divides by G*W including causal zeros.
 *   - Candidate set I = positions [0, N-W); the window is always kept.
 *   - Ties in every top-k: higher score first, then lower position.
 *   - Std is the population standard deviation.
 *   - Pooling: centred average of odd width k over I, divisor = in-range count.
 *   - Layer indices are 0-based; T averages E of layers max(0,l-m) .. l-1.
 *
 * All floating point is double.  Inputs are float32 arrays holding exact
 * values (bf16 inputs are widened exactly).  Layouts:
 *   q_win [B*W, Hq, d], k and v [T, Hkv, d] packed by cu_seqlens,
 *   per-position vectors [Hkv, T], per-(b,h) scalars [B, Hkv],
 *   budgets [B, Hkv]: keys kept by each (sequence, KV head);
 *   kept indices of (b, h) after those of every earlier pair in (b, h) order,
 *   positions relative to the sequence start, ascending, -1 padded;
 *   compacted rows per sequence: C_b + W per head, C_b = max_h budget(b, h).
 */
#ifndef BACON_REF_H
#define BACON_REF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { BACON_REF_TERM_E = 1, BACON_REF_TERM_L = 2, BACON_REF_TERM_T = 4 };

/* How the score is pooled over I before the top-K (the method does not pool;
 * the pooling and its variants are readings):
 *   MEAN_S  average pool of S = B + lambda V (default)
 *   MAX_S   max pool of S
 *   MEAN_B  average pool of B only, before calibration: pool(B) + lambda V */
enum { BACON_REF_POOL_MEAN_S = 0, BACON_REF_POOL_MAX_S = 1, BACON_REF_POOL_MEAN_B = 2 };

typedef struct {
  int num_q_heads, num_kv_heads, head_dim, window;
  int radius;         /* r of the coherence neighbourhood (paper default 5)   */
  int persist_m;      /* m, persistence depth (paper default 4)               */
  double rho;         /* scale-matching expansion (paper default 2)           */
  double gamma;       /* calibration strength (unvalued in the paper; 1)      */
  double eps;         /* stabiliser in lambda (unvalued in the paper; 1e-12)  */
  int pool_kernel;    /* odd width of the average pool of S; 1 = off          */
  int use_last_query; /* 0 = window score only (S = B)                        */
  int terms;          /* bit mask of E, L, T included in V (7 = all)          */
  int pool_mode;      /* BACON_REF_POOL_*                                     */
} bacon_ref_cfg;

/* Outputs of one layer; any pointer may be NULL to skip it. */
typedef struct {
  double *lse;                    /* [B, Hq, W] natural-log normaliser of each window row */
  double *B, *Q, *E, *L, *T, *V;  /* [Hkv, T]                                   */
  double *S;                      /* [Hkv, T] final score B + lambda V          */
  double *S_pool;                 /* [Hkv, T] pooled S on candidates, 0 elsewhere */
  double *lambda, *sigma_B, *sigma_V; /* [B, Hkv]                               */
  int32_t *m_count;               /* [B, Hkv] size of the scale-matching set    */
  int32_t *idx;                   /* kept positions, see layout above           */
  int32_t *n_kept;                /* [B, Hkv]                                   */
} bacon_ref_out;

/* Window attention of one (sequence, KV head): B and Q over n positions.
 * q(g, w) = q + g*q_head_stride + w*q_row_stride, k(i) = k + i*k_row_stride.
 * lse [group*window], attn [group*window*n] (row g*window+w) may be NULL. */
void bacon_ref_scores(int n, int window, int group, int head_dim,
                      const float *q, long q_row_stride, long q_head_stride,
                      const float *k, long k_row_stride,
                      double *lse, double *attn, double *B, double *Q);

/* E_i = [Q_i - B_i]_+ */
void bacon_ref_residual(int n, const double *B, const double *Q, double *E);

/* L = P_r E with the truncated, row-normalised neighbourhood. */
void bacon_ref_coherence(int n, int radius, const double *E, double *L);

/* T = mean of the cnt vectors prev[0..cnt-1] (each length n); 0 if cnt == 0. */
void bacon_ref_persistence(int n, int cnt, const double *const *prev, double *T);

/* Top-k of x[0..n-1] by (value desc, index asc); writes min(k,n) indices in
 * ascending order and returns their count. */
int bacon_ref_topk(int n, const double *x, int k, int32_t *out_idx);

/* AdaKV's head-wise allocation of one (layer, sequence): K_h [num_heads] from
 * the backbone score A (head h at A + h*a_stride, n_cand positions), the
 * per-head budget K and the floor fraction alpha. */
void bacon_ref_adaptive_budgets(int num_heads, int n_cand, const double *A, long a_stride,
                                int budget, double floor_alpha, int32_t *out);

/* lambda over the candidate prefix [0, n_cand) with budget K. */
double bacon_ref_lambda(int n_cand, const double *B, const double *V, int budget,
                        double rho, double gamma, double eps,
                        double *sigma_B, double *sigma_V, int32_t *m_count);

/* Centred average pool of odd width `kernel` over x[0..n-1]. */
void bacon_ref_pool(int n, int kernel, const double *x, double *out);

/* Centred max pool of odd width `kernel` over x[0..n-1] (truncated at the ends). */
void bacon_ref_pool_max(int n, int kernel, const double *x, double *out);

/* One layer of a packed batch.  budgets [batch, Hkv] are the keys kept by each
 * (sequence, KV head).  e_hist is the caller's E history [num_layers, Hkv, T];
 * layers < layer are read, layer `layer` is written.  Returns 0, or -1 on
 * invalid arguments. */
int bacon_ref_layer(const bacon_ref_cfg *cfg, int layer, int batch,
                    const int32_t *cu_seqlens, const int32_t *budgets,
                    const float *q_win, const float *k,
                    double *e_hist, bacon_ref_out *out);

/* Compacted cache of one layer: per sequence b and KV head h, rows
 * [kept positions ascending][window positions][zero rows up to C_b + W],
 * C_b = max_h budget(b, h), written to [sum_b (C_b + W), Hkv, d] with elements
 * of elem_size bytes.  budgets [batch, Hkv]. */
void bacon_ref_compact(int batch, const int32_t *cu_seqlens, const int32_t *budgets,
                       int num_kv_heads, int head_dim, int window, size_t elem_size,
                       const int32_t *idx, const int32_t *n_kept,
                       const void *k, const void *v, void *k_out, void *v_out);

/* Number of OpenMP threads used by bacon_ref_layer (0 = library default). */
void bacon_ref_set_threads(int n);
int bacon_ref_get_threads(void);

#ifdef __cplusplus
}
#endif
#endif
