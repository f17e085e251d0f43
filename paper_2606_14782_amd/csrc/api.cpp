// Host side of the C ABI declared in include/bacon.h: argument checks,
// workspace carving, layer ordering, launch sequencing and event timing.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/bacon.h"
#include "internal.h"

using namespace bacon;

namespace {

thread_local std::string g_err;

bacon_status fail(bacon_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

bacon_status hip_fail(hipError_t e, const char *what) {
  return fail(BACON_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  size_t ring, vec_b, vec_vp, vec_v, vec_pb, vec_pv, vec_s, hist_b, hist_s, list_bk, list_bp, list_bv,
      list_sk, list_sp, cnt_b, cnt_s, rec_b, rec_s, partials, lse2, lambda, hb, sb, sync, total;
  size_t sync_bytes;
  size_t vec_s_stride, hist_b_stride, hist_s_stride, hb_stride, sb_stride;   // the two copies by layer parity
  int rpad, slots;
  int64_t chunks_cap;
};

bacon_status check_shape(const bacon_shape *s) {
  if (!s) return fail(BACON_ERR_INVALID, "shape is NULL");
  if (s->num_layers < 1) return fail(BACON_ERR_INVALID, "num_layers must be >= 1");
  if (s->num_q_heads < 1 || s->num_kv_heads < 1)
    return fail(BACON_ERR_INVALID, "head counts must be >= 1");
  if (s->num_q_heads % s->num_kv_heads)
    return fail(BACON_ERR_INVALID, "num_q_heads (%d) is not a multiple of num_kv_heads (%d)",
                s->num_q_heads, s->num_kv_heads);
  if (s->window < 1) return fail(BACON_ERR_INVALID, "window must be >= 1");
  if (s->max_batch < 1) return fail(BACON_ERR_INVALID, "max_batch must be >= 1");
  if (s->max_total_tokens < 1) return fail(BACON_ERR_INVALID, "max_total_tokens must be >= 1");
  if (s->dtype != BACON_FP32 && s->dtype != BACON_BF16)
    return fail(BACON_ERR_UNSUPPORTED, "dtype %d is not supported", (int)s->dtype);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(BACON_ERR_UNSUPPORTED, "head_dim %d is not supported (64 or 128)", s->head_dim);
  if (s->max_batch > kMaxBatch)
    return fail(BACON_ERR_UNSUPPORTED, "max_batch %d exceeds %d", s->max_batch, kMaxBatch);
  const int64_t rows = (int64_t)(s->num_q_heads / s->num_kv_heads) * s->window;
  if (rows > kMaxRows)
    return fail(BACON_ERR_UNSUPPORTED, "group*window = %lld exceeds %d", (long long)rows, kMaxRows);
  if (s->max_total_tokens > ((int64_t)1 << 31) / 2)
    return fail(BACON_ERR_UNSUPPORTED, "max_total_tokens too large");
  return BACON_OK;
}

bacon_status check_params(const bacon_params *p) {
  if (p->radius < 0 || p->radius > 16) return fail(BACON_ERR_INVALID, "radius must be in [0, 16]");
  if (p->persist_m < 0 || p->persist_m > kMaxRing)
    return fail(BACON_ERR_INVALID, "persist_m must be in [0, %d]", kMaxRing);
  if (!(p->rho > 0.0) || !std::isfinite(p->rho)) return fail(BACON_ERR_INVALID, "rho must be > 0");
  if (!(p->gamma >= 0.f) || !std::isfinite(p->gamma))
    return fail(BACON_ERR_INVALID, "gamma must be >= 0");
  if (!(p->eps >= 0.f) || !std::isfinite(p->eps)) return fail(BACON_ERR_INVALID, "eps must be >= 0");
  if (p->pool_kernel < 1 || p->pool_kernel > 33 || (p->pool_kernel & 1) == 0)
    return fail(BACON_ERR_INVALID, "pool_kernel must be odd and in [1, 33]");
  if (p->use_last_query != 0 && p->use_last_query != 1)
    return fail(BACON_ERR_INVALID, "use_last_query must be 0 or 1");
  if (p->terms & ~7u) return fail(BACON_ERR_INVALID, "terms has unknown bits");
  if (p->pool_mode < BACON_POOL_MEAN_S || p->pool_mode > BACON_POOL_MEAN_B)
    return fail(BACON_ERR_INVALID, "pool_mode must be 0, 1 or 2");
  if (p->head_alloc != BACON_ALLOC_GIVEN && p->head_alloc != BACON_ALLOC_ADAPTIVE)
    return fail(BACON_ERR_INVALID, "head_alloc must be 0 or 1");
  if (!(p->alloc_floor >= 0.f && p->alloc_floor <= 1.f))
    return fail(BACON_ERR_INVALID, "alloc_floor must be in [0, 1]");
  return BACON_OK;
}

Layout layout_of(const bacon_shape *s, const bacon_params *p) {
  Layout L{};
  const int G = s->num_q_heads / s->num_kv_heads;
  L.rpad = ((G * s->window + 31) / 32) * 32;
  // E history: m + 1 slot vectors, so the slot a layer writes is never one of
  // the m its persistence term reads
  L.slots = p->persist_m + 1;
  const int tk = 32 * std::min(L.rpad / 32, 4);
  L.chunks_cap = (s->max_total_tokens + tk - 1) / tk + s->max_batch;
  const size_t vec = (size_t)s->num_kv_heads * (size_t)s->max_total_tokens * sizeof(float);
  size_t off = 0;
  L.ring = off;     off += align256((size_t)L.slots * vec);
  L.vec_b = off;    off += align256(vec);
  L.vec_vp = off;   off += align256(vec);
  L.vec_v = off;    off += align256(vec);
  L.vec_pb = off;   off += align256(vec);
  L.vec_pv = off;   off += align256(vec);
  L.vec_s_stride = align256(vec);
  L.vec_s = off;    off += 2 * L.vec_s_stride;                 // by layer parity
  const size_t hist = (size_t)s->max_batch * s->num_kv_heads * kHBins * sizeof(unsigned);
  L.hist_b_stride = align256(hist * kHCopies);
  L.hist_s_stride = align256(hist);
  L.hist_b = off;   off += 2 * L.hist_b_stride;                // by layer parity
  // meeting words of the single-read pass (arrival and done counters per
  // (sequence, KV head) on lines of their own, the error word, the published
  // row normalisers), right after the B histograms so that one clearing
  // launch covers both
  L.sync_bytes = align256((size_t)(kSyncStride * s->max_batch * s->num_kv_heads + 1) * sizeof(unsigned)) +
                 align256((size_t)s->max_batch * s->num_kv_heads * L.rpad * sizeof(unsigned));
  L.sync = off;     off += L.sync_bytes;
  L.hist_s = off;   off += 2 * L.hist_s_stride;
  L.list_bk = off;  off += align256(vec);
  L.list_bp = off;  off += align256(vec);
  L.list_bv = off;  off += align256(vec);
  L.list_sk = off;  off += align256(vec);
  L.list_sp = off;  off += align256(vec);
  const int64_t segs_cap = (s->max_total_tokens + kSegLen - 1) / kSegLen + s->max_batch;
  L.cnt_b = off;    off += align256((size_t)s->num_kv_heads * segs_cap * sizeof(int));
  L.cnt_s = off;    off += align256((size_t)s->num_kv_heads * segs_cap * sizeof(int));
  L.rec_b = off;    off += align256((size_t)s->max_batch * s->num_kv_heads * sizeof(int4));
  L.rec_s = off;    off += align256((size_t)s->max_batch * s->num_kv_heads * sizeof(int4));
  L.partials = off; off += align256((size_t)s->num_kv_heads * L.chunks_cap * L.rpad * sizeof(float2));
  L.lse2 = off;     off += align256((size_t)s->max_batch * s->num_kv_heads * L.rpad * sizeof(float));
  L.lambda = off;   off += align256((size_t)s->max_batch * s->num_kv_heads * sizeof(float));
  L.hb_stride = align256((size_t)s->max_batch * s->num_kv_heads * sizeof(int2));
  L.hb = off;       off += 2 * L.hb_stride;                   // by layer parity
  L.sb_stride = align256((size_t)s->max_batch * sizeof(int4));
  L.sb = off;       off += 2 * L.sb_stride;                   // by layer parity
  L.total = off;
  return L;
}

const char *kKernelNames[] = {"window_lse",    "lse_merge",     "window_score", "window_score_calib",
                              "segment_calib", "segment_score", "segment_cand",
                              "final_topk",    "select_calib",  "select_topk",
                              "calib_elem",    "compact",       "window_lse_kr",
                              "window_score_calib_kr", "window_score_calib_lse_kr",
                              "segment_calib_cand", "segment_score_final",
                              "window_score_calib_lse", "window_score_single", "head_alloc"};
enum KernelId { KI_LSE, KI_MERGE, KI_SCORE, KI_FUSED, KI_SEGCAL, KI_SEGSCORE, KI_SEGCAND, KI_FINAL,
                KI_SEL_CALIB, KI_SEL_TOPK, KI_ELEM, KI_COMPACT, KI_LSE_KR, KI_FUSED_KR, KI_DUAL_KR,
                KI_SEL_A, KI_SEL_B, KI_DUAL, KI_SINGLE, KI_ALLOC, KI_COUNT };

}  // namespace

struct bacon_ctx {
  bacon_shape shape;
  bacon_params params;
  char *ws;
  size_t ws_bytes;
  Layout L;
  bool prompt = false;
  int next_layer = 0;
  std::vector<int32_t> cu;
  int chunk_stages_override = 0;
  bool kr_off = false;   // key-register passes switched off (streaming passes only)
  int single_mode = -1;      // single-read pass: -1 where it pays, 0 never, 1 wherever it can run
  int single_cap = -1;       // single-read workgroups the device holds at once (-1: not yet asked)
  int cus = -1;              // compute units of the device (-1: not yet asked)
  // test instrumentation (bacon_debug_capture): per-layer copies of B, V, lambda
  float *cap_B = nullptr, *cap_V = nullptr, *cap_lambda = nullptr;
  int32_t *alloc_out = nullptr;   // [num_layers, max_batch, Hkv] budgets of the adaptive allocation
  // profiling
  bool prof = false;
  std::vector<hipEvent_t> ev_pool;
  struct Pending { int kid; hipEvent_t a, b; };
  std::vector<Pending> pending;
  size_t ev_next = 0;
  int64_t launches[KI_COUNT] = {};
  double ms[KI_COUNT] = {};
};

namespace {

// The device error word (after the meeting counters of the single-read pass):
// 1 if a meeting ran out, 2 if an allocation failed its check.
unsigned *error_word(bacon_ctx *c) {
  return reinterpret_cast<unsigned *>(c->ws + c->L.sync) +
         (size_t)kSyncStride * c->shape.max_batch * c->shape.num_kv_heads;
}

}  // namespace

namespace {

// Records events around a launch when profiling is on.
template <typename F>
bacon_status timed(bacon_ctx *c, int kid, hipStream_t s, F &&launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (c->prof && c->ev_next + 2 <= c->ev_pool.size()) {
    e0 = c->ev_pool[c->ev_next++];
    e1 = c->ev_pool[c->ev_next++];
    hipEventRecord(e0, s);
  }
  const hipError_t e = launch();
  if (e != hipSuccess) return hip_fail(e, kKernelNames[kid]);
  if (e0) {
    hipEventRecord(e1, s);
    c->pending.push_back({kid, e0, e1});
  }
  return BACON_OK;
}

bacon_status check_batch(const bacon_ctx *c, const bacon_batch *bt) {
  if (!bt) return fail(BACON_ERR_INVALID, "batch is NULL");
  if (bt->batch < 1 || bt->batch > c->shape.max_batch)
    return fail(BACON_ERR_INVALID, "batch size %d outside [1, %d]", bt->batch, c->shape.max_batch);
  if (!bt->cu_seqlens || (!bt->budgets && !bt->head_budgets))
    return fail(BACON_ERR_INVALID, "batch arrays are NULL");
  if (bt->cu_seqlens[0] != 0) return fail(BACON_ERR_INVALID, "cu_seqlens[0] must be 0");
  for (int b = 0; b < bt->batch; ++b) {
    const int64_t n = (int64_t)bt->cu_seqlens[b + 1] - bt->cu_seqlens[b];
    if (n < c->shape.window)
      return fail(BACON_ERR_INVALID, "sequence %d has %lld tokens, fewer than the window %d", b,
                  (long long)n, c->shape.window);
    if (n > kMaxSeqLen)
      return fail(BACON_ERR_UNSUPPORTED, "sequence %d has %lld tokens (max %d)", b, (long long)n,
                  kMaxSeqLen);
    if (bt->head_budgets) {
      for (int h = 0; h < c->shape.num_kv_heads; ++h)
        if (bt->head_budgets[(int64_t)b * c->shape.num_kv_heads + h] < 1)
          return fail(BACON_ERR_INVALID, "budget of sequence %d, KV head %d must be >= 1", b, h);
    } else if (bt->budgets[b] < 1) {
      return fail(BACON_ERR_INVALID, "budget of sequence %d must be >= 1", b);
    }
  }
  if (bt->cu_seqlens[bt->batch] > c->shape.max_total_tokens)
    return fail(BACON_ERR_INVALID, "total tokens %d exceed max_total_tokens %lld",
                bt->cu_seqlens[bt->batch], (long long)c->shape.max_total_tokens);
  return BACON_OK;
}

bacon_status check_prompt_batch(const bacon_ctx *c, const bacon_batch *bt) {
  if (!c->prompt) return fail(BACON_ERR_ORDER, "no prompt begun (call bacon_begin_prompt)");
  // the sequences are fixed for the prompt; the budgets may change from layer
  // to layer (a per-layer budget schedule)
  if (bt->batch + 1 != (int)c->cu.size() ||
      memcmp(bt->cu_seqlens, c->cu.data(), c->cu.size() * sizeof(int32_t)) != 0)
    return fail(BACON_ERR_INVALID, "batch sequences differ from the ones given to bacon_begin_prompt");
  return BACON_OK;
}

bacon_status check_ptr(const void *p, const char *name, size_t align) {
  if (!p) return fail(BACON_ERR_INVALID, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(p) % align)
    return fail(BACON_ERR_INVALID, "%s is not %zu-byte aligned", name, align);
  return BACON_OK;
}

#define TRY(x)                     \
  do {                             \
    bacon_status _s = (x);         \
    if (_s != BACON_OK) return _s; \
  } while (0)

// Budget of (sequence b, KV head h), and the largest budget of sequence b's
// heads (its rows per head in the compacted cache, less W).
int batch_head_budget(const bacon_batch *bt, int hkv, int b, int h) {
  return bt->head_budgets ? bt->head_budgets[(int64_t)b * hkv + h] : bt->budgets[b];
}
int batch_seq_rows(const bacon_batch *bt, int hkv, int b) {
  if (!bt->head_budgets) return bt->budgets[b];
  int m = 0;
  for (int h = 0; h < hkv; ++h) m = std::max(m, batch_head_budget(bt, hkv, b, h));
  return m;
}

// edge_tables: the split calibrate path completes L next to chunk boundaries
// from an LDS table of kEdgeEntries positions, which bounds the chunk count.
SeqTable make_table(const bacon_ctx *c, const bacon_batch *bt, int *chunk_out,
                    bool edge_tables = true, int force_chunk = 0) {
  SeqTable st{};
  st.batch = bt->batch;
  const bool bf16 = c->shape.dtype == BACON_BF16;
  const int nw = c->L.rpad / 32, tk = stage_keys(nw);
  int64_t stages = 0;
  for (int b = 0; b < bt->batch; ++b) {
    const int n = bt->cu_seqlens[b + 1] - bt->cu_seqlens[b];
    stages += (n + tk - 1) / tk;
  }
  stages *= c->shape.num_kv_heads;
  // one round of workgroups over the 256 CUs at the occupancy LDS and waves allow
  const int lds = pass_lds_bytes(PASS_FUSED, bf16, c->shape.head_dim, c->L.rpad, 4 * tk);
  const int by_lds = std::max(1, (160 * 1024) / std::max(1, lds));
  const int by_waves = std::max(1, 16 / nw);
  const int64_t slots = 256LL * std::min(by_lds, by_waves);
  int per_wg = (int)std::max<int64_t>(1, (stages + slots - 1) / slots);
  if (c->chunk_stages_override > 0) per_wg = c->chunk_stages_override;
  // the select kernel stages 2r positions around every chunk boundary
  int nmax = 0;
  for (int b = 0; b < bt->batch; ++b) nmax = std::max(nmax, bt->cu_seqlens[b + 1] - bt->cu_seqlens[b]);
  if (edge_tables && c->params.radius > 0) {
    const int min_chunk = (int)(((int64_t)nmax * 2 * c->params.radius + kEdgeEntries - 1) / kEdgeEntries);
    per_wg = std::max(per_wg, (min_chunk + tk - 1) / tk);
  }
  per_wg = std::min(per_wg, kMaxChunk / tk);
  const int chunk = force_chunk > 0 ? force_chunk : tk * per_wg;
  int cb = 0, ib = 0, kb = 0, sb = 0;
  for (int b = 0; b < bt->batch; ++b) {
    const int n = bt->cu_seqlens[b + 1] - bt->cu_seqlens[b];
    const int nseg = (n + kSegLen - 1) / kSegLen;
    st.cu[b] = bt->cu_seqlens[b];
    st.chunk_base[b] = cb;
    st.budget[b] = batch_seq_rows(bt, c->shape.num_kv_heads, b);
    st.idx_base[b] = ib;
    st.kept_base[b] = kb;
    st.seg_base[b] = sb;
    cb += (n + chunk - 1) / chunk;
    for (int h = 0; h < c->shape.num_kv_heads; ++h) ib += batch_head_budget(bt, c->shape.num_kv_heads, b, h);
    kb += st.budget[b] + c->shape.window;
    sb += nseg;
  }
  st.cu[bt->batch] = bt->cu_seqlens[bt->batch];
  st.chunk_base[bt->batch] = cb;
  st.seg_base[bt->batch] = sb;
  st.total_chunks = cb;
  st.total_segs = sb;
  *chunk_out = chunk;
  return st;
}

PassArgs pass_args(const bacon_ctx *c, const SeqTable &st, int chunk, const void *q, const void *k) {
  PassArgs a{};
  const bacon_shape &s = c->shape;
  a.q = q;
  a.k = k;
  a.Hq = s.num_q_heads;
  a.Hkv = s.num_kv_heads;
  a.G = s.num_q_heads / s.num_kv_heads;
  a.W = s.window;
  a.R = a.G * s.window;
  a.Rpad = c->L.rpad;
  a.chunk = chunk;
  a.T = s.max_total_tokens;
  a.c2 = (float)(1.4426950408889634 / std::sqrt((double)s.head_dim));
  if (c->ws) {   // a context over no workspace (the static-scratch call) sets its own
    a.partials = reinterpret_cast<float2 *>(c->ws + c->L.partials);
    a.lse2 = reinterpret_cast<float *>(c->ws + c->L.lse2);
    a.hist_B = reinterpret_cast<unsigned *>(c->ws + c->L.hist_b);
    a.ring = reinterpret_cast<float *>(c->ws + c->L.ring);
    a.vec_B = reinterpret_cast<float *>(c->ws + c->L.vec_b);
    a.vec_VP = reinterpret_cast<float *>(c->ws + c->L.vec_vp);
  }
  a.radius = c->params.radius;
  a.terms = c->params.terms;
  if (c->ws) {
    a.sync = reinterpret_cast<unsigned *>(c->ws + c->L.sync);
    a.sync_groups = c->shape.max_batch * c->shape.num_kv_heads;
    a.bcast = reinterpret_cast<unsigned *>(
        c->ws + c->L.sync + align256((size_t)(kSyncStride * a.sync_groups + 1) * sizeof(unsigned)));
  }
  (void)st;
  return a;
}

// Per-head budgets of the batch into the workspace table (budget, idx offset
// within the sequence), or NULL with one budget per sequence.  The table rides
// in the arguments of small kernels on the stream, ahead of the select.
bacon_status head_table(bacon_ctx *c, const bacon_batch *bt, hipStream_t s, const int2 **out,
                        int parity = 0) {
  *out = nullptr;
  if (!bt->head_budgets) return BACON_OK;
  const int hkv = c->shape.num_kv_heads;
  int2 *dst = reinterpret_cast<int2 *>(c->ws + c->L.hb + (size_t)parity * c->L.hb_stride);
  HbChunk ch{};
  const int n = bt->batch * hkv;
  int off = 0;
  for (int p = 0; p < n; ++p) {
    if (p % hkv == 0) off = 0;
    const int k = bt->head_budgets[p];
    ch.v[ch.n++] = make_int2(k, off);
    off += k;
    if (ch.n == kHbChunk || p == n - 1) {
      const hipError_t e = launch_set_hb(ch, dst, s);
      if (e != hipSuccess) return hip_fail(e, "budget table");
      ch.base += ch.n;
      ch.n = 0;
    }
  }
  *out = dst;
  return BACON_OK;
}

// The per-sequence budget fields (budget, idx base, kept-row base) of a
// layer's batch into the workspace table of its parity, for the launches
// that hold the jobs of two layers with different budgets.
bacon_status seq_table(bacon_ctx *c, const SeqTable &st, hipStream_t s, const int4 **out, int parity) {
  int2 *dst = reinterpret_cast<int2 *>(c->ws + c->L.sb + (size_t)parity * c->L.sb_stride);
  HbChunk ch{};
  for (int b = 0; b < st.batch; ++b) {
    ch.v[ch.n++] = make_int2(st.budget[b], st.idx_base[b]);
    ch.v[ch.n++] = make_int2(st.kept_base[b], 0);
  }
  const hipError_t e = launch_set_hb(ch, dst, s);
  if (e != hipSuccess) return hip_fail(e, "budget table");
  *out = reinterpret_cast<const int4 *>(dst);
  return BACON_OK;
}

// History slots for layer `layer`: E of layer j lives in slot j % (m + 1), so
// the previous cnt = min(m, layer) layers are the slots wr - cnt .. wr - 1
// (mod m + 1), none of them wr.
void ring_slots(const bacon_ctx *c, int layer, int *wr, int *cnt) {
  *cnt = std::min(c->params.persist_m, layer);
  *wr = layer % c->L.slots;
}

SelArgs sel_args(const bacon_ctx *c) {
  SelArgs a{};
  const bacon_shape &s = c->shape;
  const bacon_params &p = c->params;
  a.Hkv = s.num_kv_heads;
  a.W = s.window;
  a.T = s.max_total_tokens;
  a.radius = p.radius;
  a.pool_half = p.pool_kernel / 2;
  a.pool_mode = p.pool_mode;
  a.rho = p.rho;
  a.gamma = p.gamma;
  a.eps = p.eps;
  a.use_last_query = p.use_last_query;
  a.terms = p.terms;
  a.vec_B = reinterpret_cast<const float *>(c->ws + c->L.vec_b);
  a.vec_VP = reinterpret_cast<const float *>(c->ws + c->L.vec_vp);
  a.vp_chunk = 1 << 30;
  a.lambda_ws = reinterpret_cast<float *>(c->ws + c->L.lambda);
  return a;
}

int max_len(const bacon_batch *bt);

// Every workgroup of the pass must fit the LDS of one CU; checked before
// anything is enqueued.
bacon_status check_lds(const bacon_ctx *c, const bacon_batch *bt, int chunk, bool passes,
                       int sel_mode) {
  const bool bf16 = c->shape.dtype == BACON_BF16;
  if (passes && pass_lds_bytes(PASS_FUSED, bf16, c->shape.head_dim, c->L.rpad, chunk) > kLdsBytes)
    return fail(BACON_ERR_UNSUPPORTED, "pass workgroup needs more LDS than a CU has");
  if (sel_mode >= 0 && max_len(bt) > kMaxSelLen)
    return fail(BACON_ERR_UNSUPPORTED, "the split calls select sequences of up to %d tokens (%d given); "
                "the fused calls take up to %d", kMaxSelLen, max_len(bt), kMaxSeqLen);
  if (sel_mode >= 0 && select_lds_bytes(sel_mode, max_len(bt)) > (size_t)kLdsBytes)
    return fail(BACON_ERR_UNSUPPORTED, "select workgroup needs more LDS than a CU has");
  if (sel_mode == SEL_CALIB) {
    const int n = max_len(bt);
    if (chunk < n && (int64_t)((n - 1) / chunk) * 2 * c->params.radius > kEdgeEntries)
      return fail(BACON_ERR_UNSUPPORTED, "too many chunk boundaries for radius %d", c->params.radius);
  }
  return BACON_OK;
}

int max_len(const bacon_batch *bt) {
  int m = 0;
  for (int b = 0; b < bt->batch; ++b) m = std::max(m, bt->cu_seqlens[b + 1] - bt->cu_seqlens[b]);
  return m;
}

}  // namespace

extern "C" {

void bacon_default_params(bacon_params *p) {
  if (!p) return;
  p->radius = 5;
  p->persist_m = 4;
  p->rho = 2.0;
  p->gamma = 1.0f;
  p->eps = 1e-12f;
  p->pool_kernel = 7;
  p->pool_mode = BACON_POOL_MEAN_S;
  p->use_last_query = 1;
  p->terms = BACON_TERM_E | BACON_TERM_L | BACON_TERM_T;
  p->head_alloc = BACON_ALLOC_GIVEN;
  p->alloc_floor = 0.2f;
}

size_t bacon_workspace_bytes(const bacon_shape *shape, const bacon_params *params) {
  bacon_params p;
  if (params) p = *params; else bacon_default_params(&p);
  if (check_shape(shape) != BACON_OK || check_params(&p) != BACON_OK) return 0;
  return layout_of(shape, &p).total;
}

bacon_status bacon_init(bacon_ctx **ctx, const bacon_shape *shape, const bacon_params *params,
                        void *d_ws, size_t ws_bytes) {
  if (!ctx) return fail(BACON_ERR_INVALID, "ctx is NULL");
  *ctx = nullptr;
  TRY(check_shape(shape));
  bacon_params p;
  if (params) p = *params; else bacon_default_params(&p);
  TRY(check_params(&p));
  if (!d_ws) return fail(BACON_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(d_ws) % 256)
    return fail(BACON_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  const Layout L = layout_of(shape, &p);
  if (ws_bytes < L.total)
    return fail(BACON_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, L.total);
  bacon_ctx *c = new bacon_ctx();
  c->shape = *shape;
  c->params = p;
  c->ws = static_cast<char *>(d_ws);
  c->ws_bytes = ws_bytes;
  c->L = L;
  if (const char *e = std::getenv("BACON_CHUNK_STAGES")) c->chunk_stages_override = std::atoi(e);
  if (const char *e = std::getenv("BACON_KEY_REGISTERS")) c->kr_off = std::atoi(e) == 0;
  if (const char *e = std::getenv("BACON_SINGLE")) c->single_mode = std::atoi(e) == 0 ? 0 : 1;
  *ctx = c;
  return BACON_OK;
}

bacon_status bacon_free(bacon_ctx *c) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  for (hipEvent_t e : c->ev_pool) hipEventDestroy(e);
  delete c;
  return BACON_OK;
}

bacon_status bacon_begin_prompt(bacon_ctx *c, const bacon_batch *bt, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_batch(c, bt));
  c->cu.assign(bt->cu_seqlens, bt->cu_seqlens + bt->batch + 1);

  // layer 0 reads no history; the B histogram of the select starts at zero
  // (each layer's final kernel clears it for the next)
  // (each layer's final kernel clears it for the next), and so do the
  // meeting counters of the single-read pass
  const hipError_t e = launch_zero(reinterpret_cast<unsigned *>(c->ws + c->L.hist_b),
                                   (int64_t)((2 * c->L.hist_b_stride + c->L.sync_bytes) / sizeof(unsigned)),
                                   static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "clear");
  c->prompt = true;
  c->next_layer = 0;
  return BACON_OK;
}

bacon_status bacon_score(bacon_ctx *c, int32_t layer, const bacon_batch *bt, const void *d_q_win,
                         const void *d_k, float *d_lse, float *d_B, float *d_Q, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_batch(c, bt));
  if (layer < 0 || layer >= c->shape.num_layers)
    return fail(BACON_ERR_INVALID, "layer %d outside [0, %d)", layer, c->shape.num_layers);
  TRY(check_ptr(d_q_win, "q_win", 16));
  TRY(check_ptr(d_k, "k", 16));
  TRY(check_ptr(d_B, "B", 4));
  TRY(check_ptr(d_Q, "Q", 4));
  if (d_lse) TRY(check_ptr(d_lse, "lse", 4));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int chunk = 0;
  const SeqTable st = make_table(c, bt, &chunk);
  TRY(check_lds(c, bt, chunk, true, -1));
  PassArgs a = pass_args(c, st, chunk, d_q_win, d_k);
  a.T = bt->cu_seqlens[bt->batch];
  a.lse_user = d_lse;
  a.out_B = d_B;
  a.out_Q = d_Q;
  const bool bf16 = c->shape.dtype == BACON_BF16;
  const bool w32 = c->shape.window == 32;
  TRY(timed(c, KI_LSE, s, [&] { return launch_pass(PASS_LSE, bf16, c->shape.head_dim, false, a, st, s); }));
  TRY(timed(c, KI_MERGE, s, [&] { return launch_lse_merge(a, st, s); }));
  return timed(c, KI_SCORE, s, [&] { return launch_pass(PASS_SCORE, bf16, c->shape.head_dim, w32, a, st, s); });
}

bacon_status bacon_calibrate(bacon_ctx *c, int32_t layer, const bacon_batch *bt, const float *d_B,
                             const float *d_Q, float *d_S, float *d_lambda, float *d_E,
                             float *d_V, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_batch(c, bt));
  TRY(check_prompt_batch(c, bt));
  if (layer != c->next_layer)
    return fail(BACON_ERR_ORDER, "layer %d given, layer %d expected next", layer, c->next_layer);
  if (layer >= c->shape.num_layers)
    return fail(BACON_ERR_ORDER, "layer %d beyond num_layers %d", layer, c->shape.num_layers);
  TRY(check_ptr(d_B, "B", 4));
  TRY(check_ptr(d_Q, "Q", 4));
  TRY(check_ptr(d_S, "S", 4));
  TRY(check_ptr(d_lambda, "lambda", 4));
  if (d_E) TRY(check_ptr(d_E, "E", 4));
  if (d_V) TRY(check_ptr(d_V, "V", 4));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int chunk = 0;
  const SeqTable st = make_table(c, bt, &chunk);
  TRY(check_lds(c, bt, chunk, false, SEL_CALIB));
  const int64_t T = bt->cu_seqlens[bt->batch];
  ElemArgs e{};
  e.in_B = d_B;
  e.in_Q = d_Q;
  e.ring = reinterpret_cast<float *>(c->ws + c->L.ring);
  ring_slots(c, layer, &e.ring_write, &e.ring_cnt);
  e.ring_slots = c->L.slots;
  e.ring_stride = (int64_t)c->shape.num_kv_heads * T;
  e.vec_VP = reinterpret_cast<float *>(c->ws + c->L.vec_vp);
  e.Hkv = c->shape.num_kv_heads;
  e.radius = c->params.radius;
  e.chunk = chunk;
  e.T = T;
  e.terms = c->params.terms;
  // the [Hkv, T] vectors of the split path use the batch's T as row length
  TRY(timed(c, KI_ELEM, s, [&] { return launch_elem(e, st, s); }));
  SelArgs a = sel_args(c);
  a.T = T;
  a.vec_B = d_B;
  a.vp_chunk = chunk;   // same chunking as the fused pass
  a.ring = e.ring;
  a.ring_stride = e.ring_stride;
  a.ring_slot = e.ring_write;
  a.out_S = d_S;
  a.out_V = d_V;
  a.out_E = d_E;
  a.out_lambda = d_lambda;
  TRY(head_table(c, bt, s, &a.hb));
  TRY(timed(c, KI_SEL_CALIB, s, [&] { return launch_select(SEL_CALIB, max_len(bt), a, st, s); }));
  c->next_layer = layer + 1;
  return BACON_OK;
}

bacon_status bacon_select_topk(bacon_ctx *c, const bacon_batch *bt, const float *d_S,
                               int32_t *d_idx, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_batch(c, bt));
  TRY(check_ptr(d_S, "S", 4));
  TRY(check_ptr(d_idx, "idx", 4));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int chunk = 0;
  const SeqTable st = make_table(c, bt, &chunk);
  TRY(check_lds(c, bt, chunk, false, SEL_TOPK));
  SelArgs a = sel_args(c);
  a.T = bt->cu_seqlens[bt->batch];
  a.in_S = d_S;
  a.idx = d_idx;
  TRY(head_table(c, bt, s, &a.hb));
  return timed(c, KI_SEL_TOPK, s, [&] { return launch_select(SEL_TOPK, max_len(bt), a, st, s); });
}

bacon_status bacon_allocate_heads(bacon_ctx *c, const bacon_batch *bt, const float *d_B,
                                  int32_t *d_budgets, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_batch(c, bt));
  TRY(check_ptr(d_B, "B", 4));
  TRY(check_ptr(d_budgets, "budgets", 4));
  if (bt->head_budgets)
    return fail(BACON_ERR_INVALID, "the adaptive allocation takes per-sequence budgets, not head_budgets");
  if (c->shape.num_kv_heads > 32)
    return fail(BACON_ERR_UNSUPPORTED, "the adaptive allocation takes at most 32 KV heads");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int chunk = 0;
  const SeqTable st = make_table(c, bt, &chunk);
  AllocArgs a{};
  a.Hkv = c->shape.num_kv_heads;
  a.W = c->shape.window;
  a.pool_half = c->params.pool_kernel / 2;
  a.T = bt->cu_seqlens[bt->batch];
  a.alpha = c->params.alloc_floor;
  a.vec_B = d_B;
  a.vec_A = reinterpret_cast<float *>(c->ws + c->L.vec_pb);
  a.hb = reinterpret_cast<int2 *>(c->ws + c->L.hb);
  a.out = d_budgets;
  a.err = error_word(c);
  return timed(c, KI_ALLOC, s, [&] { return launch_alloc(a, st, s); });
}

bacon_status bacon_alloc_output(bacon_ctx *c, int32_t *d_budgets) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  if (d_budgets) TRY(check_ptr(d_budgets, "budgets", 4));
  c->alloc_out = d_budgets;
  return BACON_OK;
}

bacon_status bacon_compact(bacon_ctx *c, const bacon_batch *bt, const void *d_k, const void *d_v,
                           const int32_t *d_idx, void *d_k_out, void *d_v_out, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_batch(c, bt));
  TRY(check_ptr(d_k, "k", 16));
  TRY(check_ptr(d_v, "v", 16));
  TRY(check_ptr(d_idx, "idx", 4));
  TRY(check_ptr(d_k_out, "k_out", 16));
  TRY(check_ptr(d_v_out, "v_out", 16));
  hipStream_t s = static_cast<hipStream_t>(stream);
  int chunk = 0;
  const SeqTable st = make_table(c, bt, &chunk);
  CompactArgs a{};
  a.idx = d_idx;
  a.k = d_k;
  a.v = d_v;
  a.k_out = d_k_out;
  a.v_out = d_v_out;
  a.Hkv = c->shape.num_kv_heads;
  a.W = c->shape.window;
  a.row_bytes = c->shape.head_dim * (c->shape.dtype == BACON_BF16 ? 2 : 4);
  TRY(head_table(c, bt, s, &a.hb));
  return timed(c, KI_COMPACT, s, [&] { return launch_compact(a, st, s); });
}

}  // extern "C"

namespace {

// Everything the launches of one layer of the fused pass need.
struct LayerRun {
  int layer = 0;
  bool bf16 = false, w32 = false, kr = false, single = false;
  bool adaptive = false;   // head-wise budgets from the adaptive allocation
  int chunk = 0, kmax = 0;
  SeqTable st{};
  PassArgs a{};
  SegArgs g{};
  const float *lse = nullptr;   // caller normalisers (pass 1 skipped)
};

// Checks one layer's arguments and builds its launch arguments; enqueues
// nothing.  The layer order is the caller's to check.  Buffers that a layer
// of the next pair may write while this layer's select is still in flight
// (the B and S histograms and the score keys) alternate with the layer's
// parity.
bacon_status plan_layer(bacon_ctx *c, int32_t layer, const bacon_batch *bt, const void *d_q_win,
                        const void *d_k, const void *d_v, const float *d_lse, int32_t *d_idx,
                        void *d_k_out, void *d_v_out, LayerRun &r) {
  TRY(check_batch(c, bt));
  TRY(check_prompt_batch(c, bt));
  if (layer >= c->shape.num_layers)
    return fail(BACON_ERR_ORDER, "layer %d beyond num_layers %d", layer, c->shape.num_layers);
  TRY(check_ptr(d_q_win, "q_win", 16));
  TRY(check_ptr(d_k, "k", 16));
  TRY(check_ptr(d_v, "v", 16));
  TRY(check_ptr(d_idx, "idx", 4));
  TRY(check_ptr(d_k_out, "k_out", 16));
  TRY(check_ptr(d_v_out, "v_out", 16));
  r.layer = layer;
  r.lse = d_lse;
  r.bf16 = c->shape.dtype == BACON_BF16;
  r.w32 = c->shape.window == 32;
  // key-register passes where they cover the shape, else the streaming passes
  r.kr = !c->kr_off && kr_supported(r.bf16, c->shape.head_dim, c->L.rpad);
  if (r.kr) {
    r.st = make_table(c, bt, &r.chunk, false, kr_keys(r.bf16, c->shape.head_dim));
  } else {
    r.st = make_table(c, bt, &r.chunk, false);
    TRY(check_lds(c, bt, r.chunk, true, -1));
  }
  // One read of K (the single-read pass) when its meeting can complete:
  // workgroups run in grid order, chunk-major with the KV heads innermost,
  // so at most the groups of one sequence are incomplete at a time, and
  // all their chunks must fit on the GPU at once.  It pays where the whole
  // grid is resident at once and fills at least half of the GPU's slots:
  // a grid that runs in rounds stalls at every sequence split across them,
  // and a small one leaves the GPU idle through the meeting, where the two-
  // pass path overlaps two layers in each launch.  With normalisers given by
  // the caller the key-register pass 2 alone already reads K once.
  if (r.kr && !d_lse && c->single_mode != 0) {
    if (c->single_cap < 0) c->single_cap = single_resident_blocks(c->shape.head_dim, c->L.rpad);
    int nmax = 0;
    for (int b = 0; b < bt->batch; ++b) nmax = std::max(nmax, r.st.chunk_base[b + 1] - r.st.chunk_base[b]);
    const int64_t hkv = c->shape.num_kv_heads, grid = (int64_t)r.st.total_chunks * hkv;
    r.single = (int64_t)nmax * hkv <= c->single_cap &&
               (c->single_mode == 1 || (grid <= c->single_cap && 2 * grid >= c->single_cap));
  }
  r.kmax = 0;
  for (int b = 0; b < bt->batch; ++b) r.kmax = std::max(r.kmax, batch_seq_rows(bt, c->shape.num_kv_heads, b));
  r.adaptive = c->params.head_alloc == BACON_ALLOC_ADAPTIVE;
  if (r.adaptive) {
    if (bt->head_budgets)
      return fail(BACON_ERR_INVALID, "the adaptive allocation takes per-sequence budgets, not head_budgets");
    if (c->shape.num_kv_heads > 32)
      return fail(BACON_ERR_UNSUPPORTED, "the adaptive allocation takes at most 32 KV heads");
    // a head may take up to all H_kv K_b slots of its sequence, at most its candidates
    for (int b = 0; b < bt->batch; ++b) {
      const int nc = bt->cu_seqlens[b + 1] - bt->cu_seqlens[b] - c->shape.window;
      r.kmax = std::max(r.kmax, (int)std::min<int64_t>(nc, (int64_t)c->shape.num_kv_heads * bt->budgets[b]));
    }
  }
  if (final_lds_bytes(r.kmax, c->shape.window) > (size_t)kLdsBytes)
    return fail(BACON_ERR_UNSUPPORTED, "budget %d needs more LDS than a CU has", r.kmax);
  const int par = layer & 1;
  const int64_t T = bt->cu_seqlens[bt->batch];
  PassArgs &a = r.a;
  a = pass_args(c, r.st, r.chunk, d_q_win, d_k);
  a.T = T;
  a.lse_in = d_lse;
  a.hist_B += (size_t)par * c->L.hist_b_stride / sizeof(unsigned);
  int ring_cnt = 0;
  ring_slots(c, layer, &a.ring_write, &ring_cnt);
  a.ring_stride = (int64_t)c->shape.num_kv_heads * T;
  SegArgs &g = r.g;
  g = SegArgs{};
  g.Hkv = c->shape.num_kv_heads;
  g.W = c->shape.window;
  g.T = T;
  g.radius = c->params.radius;
  g.pool_half = c->params.pool_kernel / 2;
  g.pool_mode = c->params.pool_mode;
  g.vp_chunk = r.chunk;
  g.rho = c->params.rho;
  g.gamma = c->params.gamma;
  g.eps = c->params.eps;
  // B of the single-read pass is formed from probabilities stored in fp16
  // (unit roundoff 2^-11); the passes that keep them in fp32 leave B exact
  g.b_floor = r.single ? 0x1p-11f : 0.f;
  g.use_last_query = c->params.use_last_query;
  g.terms = c->params.terms;
  g.vec_B = a.vec_B;
  g.vec_VP = a.vec_VP;
  g.ring = a.ring;
  g.ring_stride = a.ring_stride;
  g.ring_slots = c->L.slots;
  g.ring_slot = a.ring_write;
  g.ring_cnt = ring_cnt;
  g.vec_V = reinterpret_cast<float *>(c->ws + c->L.vec_v);
  g.vec_pB = reinterpret_cast<float *>(c->ws + c->L.vec_pb);
  g.vec_pV = reinterpret_cast<float *>(c->ws + c->L.vec_pv);
  g.vec_S = reinterpret_cast<unsigned *>(c->ws + c->L.vec_s + (size_t)par * c->L.vec_s_stride);
  g.hist_B = a.hist_B;
  g.hist_S = reinterpret_cast<unsigned *>(c->ws + c->L.hist_s + (size_t)par * c->L.hist_s_stride);
  g.listB_key = reinterpret_cast<unsigned *>(c->ws + c->L.list_bk);
  g.listB_pos = reinterpret_cast<int *>(c->ws + c->L.list_bp);
  g.listB_v = reinterpret_cast<float *>(c->ws + c->L.list_bv);
  g.listS_key = reinterpret_cast<unsigned *>(c->ws + c->L.list_sk);
  g.listS_pos = reinterpret_cast<int *>(c->ws + c->L.list_sp);
  g.cntB = reinterpret_cast<int *>(c->ws + c->L.cnt_b);
  g.cntS = reinterpret_cast<int *>(c->ws + c->L.cnt_s);
  g.recB = reinterpret_cast<int4 *>(c->ws + c->L.rec_b);
  g.recS = reinterpret_cast<int4 *>(c->ws + c->L.rec_s);
  g.lambda_ws = reinterpret_cast<float *>(c->ws + c->L.lambda);
  g.idx = d_idx;
  g.k = d_k;
  g.v = d_v;
  g.k_out = d_k_out;
  g.v_out = d_v_out;
  g.row_bytes = c->shape.head_dim * (r.bf16 ? 2 : 4);
  g.flat_heads = r.adaptive;
  // final workgroups per (sequence, KV head): up to eight, but no more than
  // keep the launch to the rounds over the CUs that one part per head needs
  // (in a prompt call the score workgroups of the next layer share the
  // launch, one 1024-thread workgroup per CU: a batch whose score
  // workgroups alone fill the CUs takes more rounds with every part)
  if (c->cus < 0) {
    int dev = 0;
    c->cus = 256;
    if (hipGetDevice(&dev) == hipSuccess) {
      int n = 0;
      if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) c->cus = n;
    }
  }
  {
    const int hkv = c->shape.num_kv_heads, heads = std::max(1, bt->batch * hkv);
    const int score_wgs = r.st.total_segs * hkv;
    auto rounds = [&](int p) { return (score_wgs + p * heads + c->cus - 1) / c->cus; };
    int p = std::max(1, std::min(8, c->cus / heads));
    while (p > 1 && rounds(p) > rounds(1)) --p;
    g.parts = p;
  }
  return BACON_OK;
}

// The K passes of a layer.  lse_merged: its pass 1 ran with the previous
// layer's pass 2 and its normalisers are merged.  next (NULL or the next
// layer's pass 1 arguments): that pass 1 runs in this layer's pass-2 launch
// (bf16 keys; fp32 keys: in a launch right after it).
bacon_status stage_pass(bacon_ctx *c, const LayerRun &r, bool lse_merged, const PassArgs *next,
                        hipStream_t s) {
  const int d = c->shape.head_dim;
  if (r.single)
    return timed(c, KI_SINGLE, s, [&] { return launch_single(d, r.w32, r.a, r.st, s); });
  if (r.kr) {
    if (!r.lse && !lse_merged) {
      TRY(timed(c, KI_LSE_KR, s, [&] { return launch_krpass(PASS_LSE, r.bf16, d, false, r.a, r.st, s); }));
      TRY(timed(c, KI_MERGE, s, [&] { return launch_lse_merge(r.a, r.st, s); }));
    }
    if (next)
      return timed(c, KI_DUAL_KR, s, [&] { return launch_krdual(r.bf16, d, r.w32, r.a, *next, r.st, s); });
    return timed(c, KI_FUSED_KR, s, [&] { return launch_krpass(PASS_FUSED, r.bf16, d, r.w32, r.a, r.st, s); });
  }
  if (!r.lse && !lse_merged) {
    TRY(timed(c, KI_LSE, s, [&] { return launch_pass(PASS_LSE, r.bf16, d, false, r.a, r.st, s); }));
    TRY(timed(c, KI_MERGE, s, [&] { return launch_lse_merge(r.a, r.st, s); }));
  }
  if (next && r.bf16)
    return timed(c, KI_DUAL, s, [&] { return launch_pass_dual(r.bf16, d, r.w32, r.a, *next, r.st, s); });
  TRY(timed(c, KI_FUSED, s, [&] { return launch_pass(PASS_FUSED, r.bf16, d, r.w32, r.a, r.st, s); }));
  if (next)   // fp32 keys: the next layer's pass 1 in a launch of its own
    return timed(c, KI_LSE, s, [&] { return launch_pass(PASS_LSE, r.bf16, d, false, *next, r.st, s); });
  return BACON_OK;
}

// The adaptive allocation's budget table of a layer (by layer parity, where
// given head budgets go otherwise).
int2 *alloc_table(bacon_ctx *c, int layer) {
  return reinterpret_cast<int2 *>(c->ws + c->L.hb + (size_t)(layer & 1) * c->L.hb_stride);
}

// Head-wise budgets of r's layer from its window score (adaptive allocation
// only), before its calibration reads them.
bacon_status stage_alloc(bacon_ctx *c, const LayerRun &r, hipStream_t s) {
  if (!r.adaptive) return BACON_OK;
  AllocArgs a{};
  a.Hkv = c->shape.num_kv_heads;
  a.W = c->shape.window;
  a.pool_half = c->params.pool_kernel / 2;
  a.T = r.g.T;
  a.alpha = c->params.alloc_floor;
  a.vec_B = r.g.vec_B;
  a.vec_A = r.g.vec_pB;   // free until this layer's calibration writes the pooled B there
  a.hb = alloc_table(c, r.layer);
  a.out = c->alloc_out ? c->alloc_out + (size_t)r.layer * c->shape.max_batch * c->shape.num_kv_heads
                       : nullptr;
  a.sb = r.g.sb;
  a.err = error_word(c);
  return timed(c, KI_ALLOC, s, [&] { return launch_alloc(a, r.st, s); });
}

// Calibration of r's layer, with the previous layer's candidate lists and the
// next layer's row normalisers in the same launch when given.
bacon_status stage_a(bacon_ctx *c, const LayerRun &r, const LayerRun *prev, const PassArgs *next,
                     hipStream_t s) {
  if (!prev && !next) return timed(c, KI_SEGCAL, s, [&] { return launch_segcal(r.g, r.st, s); });
  return timed(c, KI_SEL_A, s, [&] {
    return launch_sel_a(r.g, prev ? &prev->g : nullptr, next, r.st, s);
  });
}

// Scores of r's layer, with the previous layer's final top-K and compaction.
bacon_status stage_b(bacon_ctx *c, const LayerRun &r, const LayerRun *prev, hipStream_t s) {
  if (!prev) return timed(c, KI_SEGSCORE, s, [&] { return launch_segscore(r.g, r.st, s); });
  return timed(c, KI_SEL_B, s, [&] { return launch_sel_b(r.g, &prev->g, r.st, prev->kmax, s); });
}

// Candidate lists, final top-K and compaction of r's layer.
bacon_status stage_tail(bacon_ctx *c, const LayerRun &r, hipStream_t s) {
  TRY(timed(c, KI_SEGCAND, s, [&] { return launch_segcand(r.g, r.st, s); }));
  return timed(c, KI_FINAL, s, [&] { return launch_segfinal(r.g, r.st, r.kmax, s); });
}

// Test instrumentation: once r's layer has its lambda (after its score
// stage), copies B, V and lambda into the capture buffers, before a later
// launch overwrites them.
bacon_status stage_capture(bacon_ctx *c, const LayerRun &r, const bacon_batch *bt, hipStream_t s) {
  if (!c->cap_B) return BACON_OK;
  const size_t vec = (size_t)c->shape.num_kv_heads * (size_t)bt->cu_seqlens[bt->batch];
  const size_t sc = (size_t)bt->batch * c->shape.num_kv_heads;
  hipError_t e = hipMemcpyAsync(c->cap_B + (size_t)r.layer * vec, r.g.vec_B, vec * sizeof(float),
                                hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->cap_V + (size_t)r.layer * vec, r.g.vec_V, vec * sizeof(float),
                       hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->cap_lambda + (size_t)r.layer * sc, r.g.lambda_ws, sc * sizeof(float),
                       hipMemcpyDeviceToDevice, s);
  return e == hipSuccess ? BACON_OK : hip_fail(e, "capture");
}

// The fused pass of one layer; d_lse (caller normalisers) skips pass 1.
bacon_status compress(bacon_ctx *c, int32_t layer, const bacon_batch *bt, const void *d_q_win,
                      const void *d_k, const void *d_v, const float *d_lse, int32_t *d_idx,
                      void *d_k_out, void *d_v_out, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  if (layer != c->next_layer)
    return fail(BACON_ERR_ORDER, "layer %d given, layer %d expected next", layer, c->next_layer);
  LayerRun r;
  TRY(plan_layer(c, layer, bt, d_q_win, d_k, d_v, d_lse, d_idx, d_k_out, d_v_out, r));
  hipStream_t s = static_cast<hipStream_t>(stream);
  TRY(head_table(c, bt, s, &r.g.hb, layer & 1));
  if (r.adaptive) r.g.hb = alloc_table(c, layer);
  TRY(stage_pass(c, r, false, nullptr, s));
  TRY(stage_alloc(c, r, s));
  TRY(stage_a(c, r, nullptr, nullptr, s));
  TRY(stage_b(c, r, nullptr, s));
  TRY(stage_capture(c, r, bt, s));
  TRY(stage_tail(c, r, s));
  c->next_layer = layer + 1;
  return BACON_OK;
}

}  // namespace

extern "C" {

bacon_status bacon_compress_layer(bacon_ctx *c, int32_t layer, const bacon_batch *bt,
                                  const void *d_q_win, const void *d_k, const void *d_v,
                                  int32_t *d_idx, void *d_k_out, void *d_v_out, void *stream) {
  return compress(c, layer, bt, d_q_win, d_k, d_v, nullptr, d_idx, d_k_out, d_v_out, stream);
}

bacon_status bacon_compress_layer_lse(bacon_ctx *c, int32_t layer, const bacon_batch *bt,
                                      const void *d_q_win, const void *d_k, const void *d_v,
                                      const float *d_lse, int32_t *d_idx, void *d_k_out,
                                      void *d_v_out, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  TRY(check_ptr(d_lse, "lse", 4));
  return compress(c, layer, bt, d_q_win, d_k, d_v, d_lse, d_idx, d_k_out, d_v_out, stream);
}

bacon_status bacon_compress_prompt(bacon_ctx *c, const bacon_batch *bt, int32_t first_layer,
                                   int32_t num_layers, const void *const *d_q_win,
                                   const void *const *d_k, const void *const *d_v,
                                   const float *const *d_lse, int32_t *const *d_idx,
                                   void *const *d_k_out, void *const *d_v_out,
                                   const bacon_batch *const *layer_batch, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  if (num_layers < 1) return fail(BACON_ERR_INVALID, "num_layers %d must be >= 1", num_layers);
  if (!d_q_win || !d_k || !d_v || !d_idx || !d_k_out || !d_v_out)
    return fail(BACON_ERR_INVALID, "a per-layer pointer array is NULL");
  if (first_layer != c->next_layer)
    return fail(BACON_ERR_ORDER, "layer %d given, layer %d expected next", first_layer, c->next_layer);
  if ((int64_t)first_layer + num_layers > c->shape.num_layers)
    return fail(BACON_ERR_ORDER, "layers %d..%d beyond num_layers %d", first_layer,
                first_layer + num_layers - 1, c->shape.num_layers);
  // every layer's arguments are checked before the first launch
  for (int i = 0; i < num_layers; ++i) {
    TRY(check_ptr(d_q_win[i], "q_win", 16));
    TRY(check_ptr(d_k[i], "k", 16));
    TRY(check_ptr(d_v[i], "v", 16));
    TRY(check_ptr(d_idx[i], "idx", 4));
    TRY(check_ptr(d_k_out[i], "k_out", 16));
    TRY(check_ptr(d_v_out[i], "v_out", 16));
    if (d_lse) TRY(check_ptr(d_lse[i], "lse", 4));
  }
  // every layer is planned (and checked) before the first launch; a layer
  // takes its own batch (budgets) when layer_batch is given
  auto lbt = [&](int i) { return layer_batch ? layer_batch[i] : bt; };
  if (layer_batch)
    for (int i = 0; i < num_layers; ++i)
      if (!layer_batch[i]) return fail(BACON_ERR_INVALID, "layer_batch[%d] is NULL", i);
  std::vector<LayerRun> runs(num_layers);
  int kmax = 0;
  for (int i = 0; i < num_layers; ++i) {
    TRY(plan_layer(c, first_layer + i, lbt(i), d_q_win[i], d_k[i], d_v[i],
                   d_lse ? d_lse[i] : nullptr, d_idx[i], d_k_out[i], d_v_out[i], runs[i]));
    kmax = std::max(kmax, runs[i].kmax);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Layers in flight at once: layer l's candidate lists run in the launch of
  // layer l+1's calibration, its final top-K and compaction in the launch of
  // layer l+1's scores (when that launch's LDS fits), and layer l+1's pass 1
  // in the launch of layer l's pass 2.  The per-head budget table of a
  // layer (if any) alternates with its parity: it is written after the
  // launch that held the final kernel of the layer two before.
  const bool overlap = sel_b_lds_bytes(kmax, c->shape.window) <= (size_t)kLdsBytes;
  bool merged = false;
  for (int i = 0; i < num_layers; ++i) {
    LayerRun &r = runs[i];
    TRY(head_table(c, lbt(i), s, &r.g.hb, r.layer & 1));
    if (r.adaptive) r.g.hb = alloc_table(c, r.layer);
    if (layer_batch) TRY(seq_table(c, r.st, s, &r.g.sb, r.layer & 1));
    const LayerRun *prev = (overlap && i > 0) ? &runs[i - 1] : nullptr;
    // the next layer's pass 1 rides in this layer's pass-2 launch, unless the
    // next layer reads K once (single-read pass) or has its normalisers given
    const PassArgs *next = (!r.lse && !r.single && i + 1 < num_layers && !runs[i + 1].single)
                               ? &runs[i + 1].a : nullptr;
    TRY(stage_pass(c, r, merged, next, s));
    TRY(stage_alloc(c, r, s));
    TRY(stage_a(c, r, prev, next, s));
    TRY(stage_b(c, r, prev, s));
    TRY(stage_capture(c, r, lbt(i), s));
    if (!overlap) TRY(stage_tail(c, r, s));
    merged = next != nullptr;
    c->next_layer = r.layer + 1;
  }
  if (overlap) TRY(stage_tail(c, runs[num_layers - 1], s));
  return BACON_OK;
}

}  // extern "C"

namespace {

// The window-row normalisers of one layer: pass 1 and the merge.  With
// scratch NULL the per-chunk partials and merged normalisers go to the
// context's workspace; otherwise to scratch (scratch_bytes long), which is
// checked before anything is enqueued.
bacon_status window_lse(bacon_ctx *c, const bacon_batch *bt, const void *d_q_win, const void *d_k,
                        float *d_lse, void *stream, char *scratch, size_t scratch_bytes,
                        bool lookup_scratch) {
  TRY(check_batch(c, bt));
  TRY(check_ptr(d_q_win, "q_win", 16));
  TRY(check_ptr(d_k, "k", 16));
  TRY(check_ptr(d_lse, "lse", 4));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf16 = c->shape.dtype == BACON_BF16;
  int chunk = 0;
  SeqTable st{};
  const bool kr = !c->kr_off && kr_supported(bf16, c->shape.head_dim, c->L.rpad);
  if (kr) {
    st = make_table(c, bt, &chunk, false, kr_keys(bf16, c->shape.head_dim));
  } else {
    st = make_table(c, bt, &chunk, false);
    TRY(check_lds(c, bt, chunk, true, -1));
  }
  PassArgs a = pass_args(c, st, chunk, d_q_win, d_k);
  a.T = bt->cu_seqlens[bt->batch];
  a.lse_user = d_lse;
  if (lookup_scratch) {
    // partials [Hkv, chunks, Rpad] float2, then the merged normalisers [B, Hkv, Rpad]
    const size_t part = align256((size_t)c->shape.num_kv_heads * st.total_chunks * c->L.rpad * sizeof(float2));
    const size_t need = part + align256((size_t)bt->batch * c->shape.num_kv_heads * c->L.rpad * sizeof(float));
    if (need > scratch_bytes)
      return fail(BACON_ERR_WORKSPACE, "the batch needs %zu bytes of scratch; the static scratch holds %zu",
                  need, scratch_bytes);
    void *p = nullptr;
    const hipError_t e = static_scratch(&p);
    if (e != hipSuccess) return hip_fail(e, "static scratch");
    scratch = static_cast<char *>(p);
    a.partials = reinterpret_cast<float2 *>(scratch);
    a.lse2 = reinterpret_cast<float *>(scratch + part);
  }
  if (kr) {
    TRY(timed(c, KI_LSE_KR, s, [&] { return launch_krpass(PASS_LSE, bf16, c->shape.head_dim, false, a, st, s); }));
  } else {
    TRY(timed(c, KI_LSE, s, [&] { return launch_pass(PASS_LSE, bf16, c->shape.head_dim, false, a, st, s); }));
  }
  TRY(timed(c, KI_MERGE, s, [&] { return launch_lse_merge(a, st, s); }));
  return BACON_OK;
}

}  // namespace

extern "C" {

bacon_status bacon_window_lse(bacon_ctx *c, const bacon_batch *bt, const void *d_q_win,
                              const void *d_k, float *d_lse, void *stream) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  return window_lse(c, bt, d_q_win, d_k, d_lse, stream, nullptr, 0, false);
}

bacon_status bacon_window_lse_static(const bacon_shape *shape, const bacon_batch *bt,
                                     const void *d_q_win, const void *d_k, float *d_lse,
                                     void *stream) {
  // a context on the stack, over no workspace: nothing is allocated
  TRY(check_shape(shape));
  bacon_ctx c;
  c.shape = *shape;
  bacon_default_params(&c.params);
  c.L = layout_of(shape, &c.params);
  c.ws = nullptr;
  c.ws_bytes = 0;
  return window_lse(&c, bt, d_q_win, d_k, d_lse, stream, nullptr, kStaticScratchBytes, true);
}

int32_t bacon_debug_device_errors(bacon_ctx *c) {
  if (!c || !c->ws) return -1;
  unsigned v = 0;
  const size_t off = c->L.sync + (size_t)kSyncStride * c->shape.max_batch * c->shape.num_kv_heads * sizeof(unsigned);
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(&v, c->ws + off, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess)
    return -1;
  return (int32_t)v;
}

bacon_status bacon_debug_capture(bacon_ctx *c, float *d_B, float *d_V, float *d_lambda) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  const int set = (d_B != nullptr) + (d_V != nullptr) + (d_lambda != nullptr);
  if (set != 0 && set != 3) return fail(BACON_ERR_INVALID, "give all three capture buffers or none");
  if (set) {
    TRY(check_ptr(d_B, "B", 4));
    TRY(check_ptr(d_V, "V", 4));
    TRY(check_ptr(d_lambda, "lambda", 4));
  }
  c->cap_B = d_B;
  c->cap_V = d_V;
  c->cap_lambda = d_lambda;
  return BACON_OK;
}

int64_t bacon_idx_count(const bacon_batch *bt, int32_t num_kv_heads) {
  if (!bt || (!bt->budgets && !bt->head_budgets) || bt->batch < 1 || num_kv_heads < 1) return 0;
  int64_t n = 0;
  for (int b = 0; b < bt->batch; ++b)
    for (int h = 0; h < num_kv_heads; ++h) n += batch_head_budget(bt, num_kv_heads, b, h);
  return n;
}

int64_t bacon_kept_rows(const bacon_batch *bt, int32_t num_kv_heads, int32_t window) {
  if (!bt || (!bt->budgets && !bt->head_budgets) || bt->batch < 1 || num_kv_heads < 1) return 0;
  int64_t n = 0;
  for (int b = 0; b < bt->batch; ++b) n += batch_seq_rows(bt, num_kv_heads, b) + window;
  return n;
}

bacon_status bacon_profile_enable(bacon_ctx *c, int32_t enable) {
  if (!c) return fail(BACON_ERR_INVALID, "ctx is NULL");
  if (enable && c->ev_pool.empty()) {
    c->ev_pool.resize(16384);
    for (auto &e : c->ev_pool) {
      // timing-only events: no system-scope cache write-back when recorded
      const hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
      if (r != hipSuccess) return hip_fail(r, "hipEventCreate");
    }
  }
  c->prof = enable != 0;
  return BACON_OK;
}

int32_t bacon_profile_read(bacon_ctx *c, bacon_kernel_time *out, int32_t max) {
  if (!c) return -1;
  for (const auto &p : c->pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      c->ms[p.kid] += ms;
      c->launches[p.kid] += 1;
    }
  }
  c->pending.clear();
  c->ev_next = 0;
  int n = 0;
  for (int k = 0; k < KI_COUNT && n < max; ++k) {
    if (!c->launches[k]) continue;
    if (out) {
      std::snprintf(out[n].name, sizeof out[n].name, "%s", kKernelNames[k]);
      out[n].launches = c->launches[k];
      out[n].total_ms = c->ms[k];
    }
    ++n;
  }
  return n;
}

const char *bacon_status_string(bacon_status s) {
  switch (s) {
    case BACON_OK: return "ok";
    case BACON_ERR_INVALID: return "invalid argument";
    case BACON_ERR_UNSUPPORTED: return "unsupported";
    case BACON_ERR_ORDER: return "layer out of order";
    case BACON_ERR_WORKSPACE: return "workspace too small";
    case BACON_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char *bacon_last_error(void) { return g_err.c_str(); }

}  // extern "C"
