/*
 * bacon_ref.c -- fp64 CPU oracle of the BACON prefill KV-compression pass.
 *
 * TEST INFRASTRUCTURE ONLY (tests, smoke check, benchmark CPU baseline).
 * Plain loops in double precision, following the paper's steps in order;
 * no blocking, fusion or reordering.  The only parallelism is an OpenMP
 * loop over independent (sequence, KV head) pairs of a layer.
 */
#include "bacon_ref.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ---------------------------------------------------------------------- */
/* Sec. 4.1, Eq. window_score and Sec. 4.2, Eq. last_query_score.
 * A_{q,i} = softmax over keys i <= q of q.k_i / sqrt(d)   (App. A).
 * Window rows are the last W positions t_w = n - W + w; D = n - 1 is row W-1.
 * With GQA the G query heads of the KV head are averaged (reading). */
void bacon_ref_scores(int n, int window, int group, int head_dim,
                      const float *q, long q_row_stride, long q_head_stride,
                      const float *k, long k_row_stride,
                      double *lse, double *attn, double *B, double *Q) {
  double *s = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  const double scale = 1.0 / sqrt((double)head_dim);
  for (int i = 0; i < n; ++i) { B[i] = 0.0; Q[i] = 0.0; }
  for (int g = 0; g < group; ++g) {
    for (int w = 0; w < window; ++w) {
      const float *qv = q + (long)g * q_head_stride + (long)w * q_row_stride;
      const int t = n - window + w;          /* position of this query row */
      /* logits of the causal row */
      for (int i = 0; i <= t; ++i) {
        const float *kv = k + (long)i * k_row_stride;
        double dot = 0.0;
        for (int c = 0; c < head_dim; ++c) dot += (double)qv[c] * (double)kv[c];
        s[i] = dot * scale;
      }
      double mx = -INFINITY;
      for (int i = 0; i <= t; ++i) if (s[i] > mx) mx = s[i];
      double z = 0.0;
      for (int i = 0; i <= t; ++i) z += exp(s[i] - mx);
      const double l = mx + log(z);
      if (lse) lse[g * window + w] = l;
      double *arow = attn ? attn + ((long)g * window + w) * n : NULL;
      for (int i = 0; i < n; ++i) {
        const double a = (i <= t) ? exp(s[i] - l) : 0.0;
        B[i] += a;
        if (w == window - 1) Q[i] += a;
        if (arow) arow[i] = a;
      }
    }
  }
  const double inv_b = 1.0 / ((double)group * (double)window);
  const double inv_q = 1.0 / (double)group;
  for (int i = 0; i < n; ++i) { B[i] *= inv_b; Q[i] *= inv_q; }
  free(s);
}

/* Sec. 4.2, Eq. boundary_residual: E = [Q - B]_+ (a select keeps +0). */
void bacon_ref_residual(int n, const double *B, const double *Q, double *E) {
  for (int i = 0; i < n; ++i) E[i] = (Q[i] > B[i]) ? (Q[i] - B[i]) : 0.0;
}

/* Sec. 4.3, Eqs. neighbor_matrix and intra_layer_coherence:
 * N_r(i) = {u : |u - i| <= r, u inside the sequence}, (P_r)_{i,u} = 1/|N_r(i)|. */
void bacon_ref_coherence(int n, int radius, const double *E, double *L) {
  for (int i = 0; i < n; ++i) {
    const int lo = (i - radius < 0) ? 0 : i - radius;
    const int hi = (i + radius > n - 1) ? n - 1 : i + radius;
    double acc = 0.0;
    for (int u = lo; u <= hi; ++u) acc += E[u];
    L[i] = acc / (double)(hi - lo + 1);
  }
}

/* Sec. 4.3, Eq. inter_layer_persistence: mean of E over the preceding
 * layers of the causal set; 0 when the set is empty. */
void bacon_ref_persistence(int n, int cnt, const double *const *prev, double *T) {
  for (int i = 0; i < n; ++i) {
    if (cnt == 0) { T[i] = 0.0; continue; }
    double acc = 0.0;
    for (int j = 0; j < cnt; ++j) acc += prev[j][i];
    T[i] = acc / (double)cnt;
  }
}

/* TopK with the tie rule (score desc, position asc), via a full sort. */
typedef struct { double v; int32_t i; } vi_pair;

static int cmp_desc(const void *a, const void *b) {
  const vi_pair *x = (const vi_pair *)a, *y = (const vi_pair *)b;
  if (x->v > y->v) return -1;
  if (x->v < y->v) return 1;
  return (x->i < y->i) ? -1 : (x->i > y->i);
}

static int cmp_int(const void *a, const void *b) {
  const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x < y) ? -1 : (x > y);
}

int bacon_ref_topk(int n, const double *x, int k, int32_t *out_idx) {
  if (n <= 0 || k <= 0) return 0;
  vi_pair *p = (vi_pair *)malloc(sizeof(vi_pair) * (size_t)n);
  for (int i = 0; i < n; ++i) { p[i].v = x[i]; p[i].i = i; }
  qsort(p, (size_t)n, sizeof(vi_pair), cmp_desc);
  const int cnt = (k < n) ? k : n;
  for (int j = 0; j < cnt; ++j) out_idx[j] = p[j].i;
  qsort(out_idx, (size_t)cnt, sizeof(int32_t), cmp_int);
  free(p);
  return cnt;
}

/* App. B, AdaKV as the backbone: its head-wise budget allocation for one
 * (layer, sequence), kept unchanged under BACON (App. B, Implementation
 * Details).  Read here as AdaKV's published rule: every KV head keeps its top
 * f = floor(alpha K) positions by the backbone score A; the other H (K - f)
 * slots of the layer's budget go to the highest scores over the union of
 * every head's remaining positions (ties: score desc, head asc, position
 * asc); K_h = f + the head's share of the union.  With K >= n_cand every head
 * keeps all its candidates, and K_h = K. */
typedef struct { double v; int32_t h, i; } hvi;

static int cmp_union(const void *a, const void *b) {
  const hvi *x = (const hvi *)a, *y = (const hvi *)b;
  if (x->v > y->v) return -1;
  if (x->v < y->v) return 1;
  if (x->h != y->h) return (x->h < y->h) ? -1 : 1;
  return (x->i < y->i) ? -1 : (x->i > y->i);
}

void bacon_ref_adaptive_budgets(int num_heads, int n_cand, const double *A, long a_stride,
                                int budget, double floor_alpha, int32_t *out) {
  if (budget >= n_cand) {
    for (int h = 0; h < num_heads; ++h) out[h] = budget;
    return;
  }
  long ff = (long)floor(floor_alpha * (double)budget);
  if (ff < 0) ff = 0;
  if (ff > budget) ff = budget;
  const int f = (int)ff;
  /* the union: every head's positions after its own top f */
  hvi *u = (hvi *)malloc(sizeof(hvi) * (size_t)num_heads * (size_t)n_cand);
  vi_pair *p = (vi_pair *)malloc(sizeof(vi_pair) * (size_t)n_cand);
  long nu = 0;
  for (int h = 0; h < num_heads; ++h) {
    for (int i = 0; i < n_cand; ++i) { p[i].v = A[h * a_stride + i]; p[i].i = i; }
    qsort(p, (size_t)n_cand, sizeof(vi_pair), cmp_desc);
    for (int j = f; j < n_cand; ++j) {
      u[nu].v = p[j].v;
      u[nu].h = h;
      u[nu].i = p[j].i;
      ++nu;
    }
  }
  qsort(u, (size_t)nu, sizeof(hvi), cmp_union);
  const long R = (long)num_heads * (long)(budget - f);
  for (int h = 0; h < num_heads; ++h) out[h] = f;
  for (long j = 0; j < R && j < nu; ++j) out[u[j].h] += 1;
  free(p);
  free(u);
}

/* Sec. 4.4: M = min(rho K, |I|) (Eq. scale_matching_size), the scale-matching
 * set = TopK of B over I (Eq. scale_matching_set), and the closed-form
 * minimiser lambda = gamma Std(B) / (Std(V) + eps) (Eq. lambda_solution). */
double bacon_ref_lambda(int n_cand, const double *B, const double *V, int budget,
                        double rho, double gamma, double eps,
                        double *sigma_B, double *sigma_V, int32_t *m_count) {
  long mm = (long)floor(rho * (double)budget);
  if (mm > n_cand) mm = n_cand;
  if (mm < 0) mm = 0;
  const int M = (int)mm;
  if (m_count) *m_count = M;
  if (M == 0) {
    if (sigma_B) *sigma_B = 0.0;
    if (sigma_V) *sigma_V = 0.0;
    return 0.0;
  }
  int32_t *sel = (int32_t *)malloc(sizeof(int32_t) * (size_t)M);
  bacon_ref_topk(n_cand, B, M, sel);
  /* Population variance, two-pass; values are first shifted by the first
   * member of the set (variance is shift-invariant), so constant data gives
   * exactly 0 rather than rounding noise that eps would amplify. */
  const double b0 = B[sel[0]], v0 = V[sel[0]];
  double mb = 0.0, mv = 0.0;
  for (int j = 0; j < M; ++j) { mb += B[sel[j]] - b0; mv += V[sel[j]] - v0; }
  mb /= (double)M;
  mv /= (double)M;
  double vb = 0.0, vv = 0.0;
  for (int j = 0; j < M; ++j) {
    const double db = (B[sel[j]] - b0) - mb, dv = (V[sel[j]] - v0) - mv;
    vb += db * db;
    vv += dv * dv;
  }
  free(sel);
  const double sb = sqrt(vb / (double)M), sv = sqrt(vv / (double)M);
  if (sigma_B) *sigma_B = sb;
  if (sigma_V) *sigma_V = sv;
  return gamma * sb / (sv + eps);
}

/* Average pool of S over the candidates (SnapKV convention, reading). */
void bacon_ref_pool(int n, int kernel, const double *x, double *out) {
  const int half = kernel / 2;
  for (int i = 0; i < n; ++i) {
    const int lo = (i - half < 0) ? 0 : i - half;
    const int hi = (i + half > n - 1) ? n - 1 : i + half;
    double acc = 0.0;
    for (int u = lo; u <= hi; ++u) acc += x[u];
    out[i] = acc / (double)(hi - lo + 1);
  }
}

/* Max pool of S over the candidates (the max-pooling variant, reading). */
void bacon_ref_pool_max(int n, int kernel, const double *x, double *out) {
  const int half = kernel / 2;
  for (int i = 0; i < n; ++i) {
    const int lo = (i - half < 0) ? 0 : i - half;
    const int hi = (i + half > n - 1) ? n - 1 : i + half;
    double mx = x[lo];
    for (int u = lo + 1; u <= hi; ++u)
      if (x[u] > mx) mx = x[u];
    out[i] = mx;
  }
}

static int g_threads = 0;
void bacon_ref_set_threads(int n) { g_threads = n; }
int bacon_ref_get_threads(void) {
#ifdef _OPENMP
  return g_threads > 0 ? g_threads : omp_get_max_threads();
#else
  return 1;
#endif
}

/* One (sequence, KV head) of one layer: every step in the paper's order. */
static void one_head(const bacon_ref_cfg *c, int layer, int b, int h, int batch,
                     const int32_t *cu, const int32_t *budgets, const long *idx_off,
                     const float *q_win, const float *k, double *e_hist, long T,
                     bacon_ref_out *o) {
  const int Hq = c->num_q_heads, Hkv = c->num_kv_heads, d = c->head_dim, W = c->window;
  const int G = Hq / Hkv;
  const int n = cu[b + 1] - cu[b];
  const long off = (long)h * T + cu[b];
  const int n_cand = n - W;              /* candidate set I = [0, n - W) */
  const int K = budgets[(long)b * Hkv + h];     /* budget of this (sequence, KV head) */
  (void)batch;

  double *B = (double *)malloc(sizeof(double) * (size_t)n);
  double *Q = (double *)malloc(sizeof(double) * (size_t)n);
  double *E = e_hist + (long)layer * Hkv * T + off;   /* this layer's E, kept for later T */
  double *L = (double *)malloc(sizeof(double) * (size_t)n);
  double *Tv = (double *)malloc(sizeof(double) * (size_t)n);
  double *V = (double *)malloc(sizeof(double) * (size_t)n);
  double *S = (double *)malloc(sizeof(double) * (size_t)n);
  double *P = (double *)malloc(sizeof(double) * (size_t)(n_cand > 0 ? n_cand : 1));
  double *lse = (double *)malloc(sizeof(double) * (size_t)G * W);

  /* a1/a2: causal window attention, averaged over the window and the group */
  const float *qb = q_win + ((long)b * W * Hq + (long)h * G) * d;
  const float *kb = k + ((long)cu[b] * Hkv + h) * d;
  bacon_ref_scores(n, W, G, d, qb, (long)Hq * d, (long)d, kb, (long)Hkv * d, lse, NULL, B, Q);

  /* a3: residual, coherence, persistence, calibrated evidence */
  bacon_ref_residual(n, B, Q, E);
  bacon_ref_coherence(n, c->radius, E, L);
  const int cnt = (layer < c->persist_m) ? layer : c->persist_m;
  const double *prev[64];
  for (int j = 0; j < cnt; ++j) prev[j] = e_hist + (long)(layer - cnt + j) * Hkv * T + off;
  bacon_ref_persistence(n, cnt, prev, Tv);
  for (int i = 0; i < n; ++i)
    V[i] = ((c->terms & BACON_REF_TERM_E) ? E[i] : 0.0) +
           ((c->terms & BACON_REF_TERM_L) ? L[i] : 0.0) +
           ((c->terms & BACON_REF_TERM_T) ? Tv[i] : 0.0);

  /* a4: variance-matched lambda over the top-rho*K window scores */
  double sb = 0.0, sv = 0.0, lam = 0.0;
  int32_t mcount = 0;
  const int nc = n_cand > 0 ? n_cand : 0;
  lam = bacon_ref_lambda(nc, B, V, K, c->rho, c->gamma, c->eps, &sb, &sv, &mcount);
  if (!c->use_last_query) lam = 0.0;

  /* a5: final score (Eq. bacon_score), pooling over I, top-K */
  for (int i = 0; i < n; ++i) S[i] = B[i] + lam * V[i];
  if (nc > 0) {
    if (c->pool_mode == BACON_REF_POOL_MAX_S) {
      bacon_ref_pool_max(nc, c->pool_kernel, S, P);
    } else if (c->pool_mode == BACON_REF_POOL_MEAN_B) {
      /* pooling before calibration: the window score is pooled, V is not */
      bacon_ref_pool(nc, c->pool_kernel, B, P);
      for (int i = 0; i < nc; ++i) P[i] += lam * V[i];
    } else {
      bacon_ref_pool(nc, c->pool_kernel, S, P);
    }
  }
  int32_t *idx_out = o->idx ? o->idx + idx_off[(long)b * Hkv + h] : NULL;
  int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)(K > 0 ? K : 1));
  const int kept = bacon_ref_topk(nc, P, K, tmp);
  if (idx_out) {
    for (int j = 0; j < K; ++j) idx_out[j] = (j < kept) ? tmp[j] : -1;
  }
  free(tmp);

  /* outputs */
  const long so = (long)b * Hkv + h;
  if (o->lse)
    for (int g = 0; g < G; ++g)
      for (int w = 0; w < W; ++w)
        o->lse[((long)b * Hq + (long)h * G + g) * W + w] = lse[g * W + w];
  if (o->B) memcpy(o->B + off, B, sizeof(double) * (size_t)n);
  if (o->Q) memcpy(o->Q + off, Q, sizeof(double) * (size_t)n);
  if (o->E) memcpy(o->E + off, E, sizeof(double) * (size_t)n);
  if (o->L) memcpy(o->L + off, L, sizeof(double) * (size_t)n);
  if (o->T) memcpy(o->T + off, Tv, sizeof(double) * (size_t)n);
  if (o->V) memcpy(o->V + off, V, sizeof(double) * (size_t)n);
  if (o->S) memcpy(o->S + off, S, sizeof(double) * (size_t)n);
  if (o->S_pool)
    for (int i = 0; i < n; ++i) o->S_pool[off + i] = (i < nc) ? P[i] : 0.0;
  if (o->lambda) o->lambda[so] = lam;
  if (o->sigma_B) o->sigma_B[so] = sb;
  if (o->sigma_V) o->sigma_V[so] = sv;
  if (o->m_count) o->m_count[so] = mcount;
  if (o->n_kept) o->n_kept[so] = kept;

  free(B); free(Q); free(L); free(Tv); free(V); free(S); free(P); free(lse);
}

int bacon_ref_layer(const bacon_ref_cfg *c, int layer, int batch,
                    const int32_t *cu, const int32_t *budgets,
                    const float *q_win, const float *k,
                    double *e_hist, bacon_ref_out *o) {
  if (!c || !cu || !budgets || !q_win || !k || !e_hist || !o) return -1;
  if (batch < 1 || layer < 0 || c->num_kv_heads < 1 || c->num_q_heads % c->num_kv_heads)
    return -1;
  if (c->window < 1 || c->head_dim < 1 || c->radius < 0 || c->persist_m < 0 ||
      c->persist_m > 64 || c->pool_kernel < 1 || (c->pool_kernel & 1) == 0 ||
      c->pool_mode < BACON_REF_POOL_MEAN_S || c->pool_mode > BACON_REF_POOL_MEAN_B)
    return -1;
  const int pairs = batch * c->num_kv_heads;
  for (int b = 0; b < batch; ++b)
    if (cu[b + 1] - cu[b] < c->window) return -1;
  /* a budget may be 0 (a head-wise allocation such as AdaKV's, App. B, can
   * leave a head without slots): that head keeps no position */
  for (int p = 0; p < pairs; ++p)
    if (budgets[p] < 0) return -1;
  const long T = cu[batch];
  /* kept indices of (b, h) start after those of every earlier pair */
  long *idx_off = (long *)malloc(sizeof(long) * (size_t)(pairs + 1));
  idx_off[0] = 0;
  for (int p = 0; p < pairs; ++p) idx_off[p + 1] = idx_off[p] + budgets[p];
#ifdef _OPENMP
  const int nt = bacon_ref_get_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
#endif
  for (int p = 0; p < pairs; ++p) {
    one_head(c, layer, p / c->num_kv_heads, p % c->num_kv_heads, batch, cu, budgets,
             idx_off, q_win, k, e_hist, T, o);
  }
  free(idx_off);
  return 0;
}

/* Cache construction (after Eq. topk_selection): keep the selected rows and
 * the window rows, in ascending position. */
void bacon_ref_compact(int batch, const int32_t *cu, const int32_t *budgets,
                       int Hkv, int d, int W, size_t es,
                       const int32_t *idx, const int32_t *n_kept,
                       const void *k, const void *v, void *k_out, void *v_out) {
  const size_t row = (size_t)d * es;
  long out_row0 = 0, idx0 = 0;
  for (int b = 0; b < batch; ++b) {
    const int n = cu[b + 1] - cu[b];
    /* rows per head of this sequence: the largest budget of its heads, plus W */
    int C = 0;
    for (int h = 0; h < Hkv; ++h)
      if (budgets[(long)b * Hkv + h] > C) C = budgets[(long)b * Hkv + h];
    for (int h = 0; h < Hkv; ++h) {
      const int K = budgets[(long)b * Hkv + h];
      const int kept = n_kept[(long)b * Hkv + h];
      const int32_t *ib = idx + idx0;
      idx0 += K;
      for (int j = 0; j < C + W; ++j) {
        long src = -1;
        if (j < kept) src = ib[j];
        else if (j < kept + W) src = n - W + (j - kept);
        const size_t dst = ((size_t)(out_row0 + j) * Hkv + h) * row;
        if (src < 0) {
          memset((char *)k_out + dst, 0, row);
          memset((char *)v_out + dst, 0, row);
        } else {
          const size_t s = ((size_t)(cu[b] + src) * Hkv + h) * row;
          memcpy((char *)k_out + dst, (const char *)k + s, row);
          memcpy((char *)v_out + dst, (const char *)v + s, row);
        }
      }
    }
    out_row0 += C + W;
  }
}
