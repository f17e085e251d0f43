// gfx950 kernels of the BACON prefill KV-compression pass.
//
// Pass 1 (PASS_LSE) and pass 2 (PASS_SCORE / PASS_FUSED) stream the layer's
// keys once each.  A workgroup owns one (KV head, key chunk); its waves own
// the 32-row tiles of the G*W window queries of that KV head.  Key tiles are
// staged through LDS with coalesced 16-byte loads and consumed by 32x32 MFMA
// (bf16: v_mfma_f32_32x32x16_bf16, fp32: v_mfma_f32_32x32x2_f32).
//
//  * Pass 1 computes D = K Q^T so each lane holds one query row: the running
//    row max and sum of exp2 stay in-lane; per-chunk partials are merged by
//    the last workgroup of each (sequence, KV head) into the row normaliser.
//  * Pass 2 computes D = Q K^T so each lane holds one key: the window mean B
//    and last-query score Q are in-lane sums over the lane's rows, reduced
//    across row tiles through LDS in a fixed order (deterministic).  The fused
//    variant then forms E = [Q-B]_+ (Eq. boundary_residual), reads the E of
//    the previous layers for T (Eq. inter_layer_persistence) and appends E to
//    the history ring.
//
// The select kernel (one workgroup per (sequence, KV head)) computes
// L = P_r E (Eq. intra_layer_coherence), V (Eq. structurally_calibrated_evidence),
// the scale-matching set and lambda (Eqs. scale_matching_set, lambda_solution),
// S (Eq. bacon_score), the pooled score, the top-K (Eq. topk_selection) and
// optionally gathers the compacted cache.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace bacon {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr float kLn2 = 0.69314718055994531f;

// ---------------------------------------------------------------- MFMA units
// A "unit" is 16 bytes per lane: 8 bf16 (one 32x32x16 step) or 4 fp32 (four
// 32x32x2 steps).  Lane l holds row/column l%32 and the k-slice chosen by l/32;
// the same dimension permutation is used for both operands, so any slicing
// of d gives the exact dot product.
template <bool BF16>
__device__ __forceinline__ f32x16 mfma_unit(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (BF16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  } else {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
}

// Row (or column) of accumulator register `reg` in the 32x32 output layout.
__device__ __forceinline__ int acc_row(int reg, int half) {
  return 8 * (reg >> 2) + 4 * half + (reg & 3);
}

__device__ __forceinline__ int find_seq(const SeqTable &st, int chunk) {
  int b = 0;
  while (b + 1 < st.batch && st.chunk_base[b + 1] <= chunk) ++b;
  return b;
}

// ---------------------------------------------------------------- passes
template <bool BF16, int D>
struct PassCfg {
  static constexpr int ES = BF16 ? 2 : 4;
  static constexpr int ROWB = D * ES;          // bytes per key / query row
  static constexpr int NU = ROWB / 32;         // 16-byte units per lane
  static constexpr int PIECES = ROWB / 16;     // 16-byte pieces per row
  static constexpr int STRIDE = ROWB + 16;     // padded LDS row (bank spread)
  static constexpr int MAXL = PIECES / 2;      // max staged loads per thread
};

__host__ __device__ inline int stage_keys(int nw) { return 32 * (nw < 4 ? nw : 4); }

template <int MODE, bool BF16, int D, bool W32>
__global__ __launch_bounds__(512) void k_pass(PassArgs a, SeqTable st) {
  using C = PassCfg<BF16, D>;
  extern __shared__ __align__(16) unsigned char smem[];
  const int nw = blockDim.x >> 6;
  const int nt = blockDim.x;
  const int tk = stage_keys(nw);
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63, half = lane >> 5, l32 = lane & 31;
  const int h = blockIdx.y;
  const int gchunk = blockIdx.x;
  const int b = find_seq(st, gchunk);
  const int c = gchunk - st.chunk_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int k0 = c * a.chunk;
  const int k1 = min(n, k0 + a.chunk);
  const int W = a.W;
  const int wfirst = n - W;                      // position of window row 0

  unsigned char *kbuf = smem;
  float *red = reinterpret_cast<float *>(smem + 2 * tk * C::STRIDE);  // [2][2][nw][tk]

  // Query fragments of this wave's row tile.
  u32x4 qf[C::NU];
  {
    const int r = wave * 32 + l32;
    if (r < a.R) {
      const int g = r / W, w = r - g * W;
      const unsigned char *qp = static_cast<const unsigned char *>(a.q) +
          ((int64_t)(b * W + w) * a.Hq + (int64_t)h * a.G + g) * C::ROWB + 16 * half;
#pragma unroll
      for (int u = 0; u < C::NU; ++u) qf[u] = *reinterpret_cast<const u32x4 *>(qp + 32 * u);
    } else {
#pragma unroll
      for (int u = 0; u < C::NU; ++u) qf[u] = u32x4{0u, 0u, 0u, 0u};
    }
  }

  // Stage loader: thread t moves pieces q = t + j*nt of the stage.
  const unsigned char *kb = static_cast<const unsigned char *>(a.k) +
                            ((int64_t)st.cu[b] * a.Hkv + h) * C::ROWB;
  const int64_t kstride = (int64_t)a.Hkv * C::ROWB;
  const int stage_pieces = tk * C::PIECES;
  const int loads = (stage_pieces + nt - 1) / nt;
  u32x4 pre[C::MAXL];
  auto fetch = [&](int s) {
    const int key0 = k0 + s * tk;
    const int nvalid = min(tk, k1 - key0);
#pragma unroll
    for (int j = 0; j < C::MAXL; ++j) {
      if (j < loads) {
        const int q = t + j * nt;
        const int key = q / C::PIECES, piece = q % C::PIECES;
        if (q < stage_pieces && key < nvalid)
          pre[j] = *reinterpret_cast<const u32x4 *>(kb + (int64_t)(key0 + key) * kstride + 16 * piece);
        else
          pre[j] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto commit = [&](int buf) {
    unsigned char *dst = kbuf + buf * tk * C::STRIDE;
#pragma unroll
    for (int j = 0; j < C::MAXL; ++j) {
      if (j < loads) {
        const int q = t + j * nt;
        if (q < stage_pieces) {
          const int key = q / C::PIECES, piece = q % C::PIECES;
          *reinterpret_cast<u32x4 *>(dst + key * C::STRIDE + 16 * piece) = pre[j];
        }
      }
    }
  };

  const int nstages = (k1 - k0 + tk - 1) / tk;

  // ---- pass-1 state: running max (raw logit units) and sum of exp2
  float m_run = -INFINITY, l_run = 0.f;
  int tpos_row = 0;                // position of this lane's query row
  {
    const int r = wave * 32 + l32;
    tpos_row = wfirst + (r < a.R ? r % W : W - 1);
  }
  // ---- pass-2 state
  float nl[16];                    // -lse2 of the lane's 16 rows
  int wrow[16];                    // window index of each row (W for pad rows)
  uint32_t lastmask = 0;           // rows that are the last query of their head
  if constexpr (MODE != PASS_LSE) {
    const float *l2 = a.lse2 + ((int64_t)b * a.Hkv + h) * a.Rpad;
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int r = wave * 32 + acc_row(reg, half);
      nl[reg] = -l2[r];
      wrow[reg] = (r < a.R) ? r % W : W;
      if (!W32 && r < a.R && (r % W) == W - 1) lastmask |= 1u << reg;
    }
  }

  fetch(0);
  commit(0);
  __syncthreads();
  for (int s = 0; s < nstages; ++s) {
    const int buf = s & 1;
    if (s + 1 < nstages) fetch(s + 1);
    const unsigned char *kl = kbuf + buf * tk * C::STRIDE;
    const int ntile = min(tk, k1 - (k0 + s * tk));
#pragma unroll 1
    for (int kt = 0; kt * 32 < ntile; ++kt) {
      const int kbase = k0 + s * tk + kt * 32;   // first key of the tile (sequence-relative)
      const unsigned char *kr = kl + (kt * 32 + l32) * C::STRIDE + 16 * half;
      f32x16 acc = {};
      if constexpr (MODE == PASS_LSE) {
#pragma unroll
        for (int u = 0; u < C::NU; ++u)
          acc = mfma_unit<BF16>(*reinterpret_cast<const u32x4 *>(kr + 32 * u), qf[u], acc);
        // acc[reg]: key kbase + acc_row(reg, half), row = wave*32 + l32
        const bool edge = (kbase + 31 >= k1) || (kbase + 31 > wfirst);
        if (edge) {
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) {
            const int key = kbase + acc_row(reg, half);
            if (!(key < k1 && key <= tpos_row)) acc[reg] = -INFINITY;
          }
        }
        float mt = acc[0];
#pragma unroll
        for (int reg = 1; reg < 16; ++reg) mt = fmaxf(mt, acc[reg]);
        if (mt > m_run) {
          l_run *= __builtin_amdgcn_exp2f((m_run - mt) * a.c2);
          m_run = mt;
        }
        if (m_run != -INFINITY) {
          const float off = -m_run * a.c2;
          float sum = 0.f;
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) sum += __builtin_amdgcn_exp2f(fmaf(acc[reg], a.c2, off));
          l_run += sum;
        }
      } else {
#pragma unroll
        for (int u = 0; u < C::NU; ++u)
          acc = mfma_unit<BF16>(qf[u], *reinterpret_cast<const u32x4 *>(kr + 32 * u), acc);
        // acc[reg]: row wave*32 + acc_row(reg, half), key kbase + l32
        float p[16];
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) p[reg] = __builtin_amdgcn_exp2f(fmaf(acc[reg], a.c2, nl[reg]));
        const int key = kbase + l32;
        const bool edge = (kbase + 31 >= k1) || (kbase + 31 > wfirst);
        if (edge) {
#pragma unroll
          for (int reg = 0; reg < 16; ++reg)
            if (!(key < k1 && key - wfirst <= wrow[reg])) p[reg] = 0.f;
        }
        float bs = 0.f, qs = 0.f;
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) bs += p[reg];
        if constexpr (W32) {
          qs = half ? p[15] : 0.f;
        } else {
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) qs += ((lastmask >> reg) & 1u) ? p[reg] : 0.f;
        }
        bs += __shfl_xor(bs, 32);
        qs += __shfl_xor(qs, 32);
        if (half == 0) {
          float *rb = red + ((buf * 2 + 0) * nw + wave) * tk;
          float *rq = red + ((buf * 2 + 1) * nw + wave) * tk;
          rb[kt * 32 + l32] = bs;
          rq[kt * 32 + l32] = qs;
        }
      }
    }
    if (s + 1 < nstages) commit(buf ^ 1);
    __syncthreads();
    if constexpr (MODE != PASS_LSE) {
      // Epilogue of stage s: fixed-order reduction over row tiles.
      if (t < ntile) {
        const float *rb = red + (buf * 2 + 0) * nw * tk;
        const float *rq = red + (buf * 2 + 1) * nw * tk;
        float sb = 0.f, sq = 0.f;
        for (int w = 0; w < nw; ++w) {
          sb += rb[w * tk + t];
          sq += rq[w * tk + t];
        }
        const float Bv = sb / (float)(a.G * W);
        const float Qv = sq / (float)a.G;
        const int64_t pos = (int64_t)h * a.T + st.cu[b] + k0 + s * tk + t;
        if constexpr (MODE == PASS_SCORE) {
          a.out_B[pos] = Bv;
          a.out_Q[pos] = Qv;
        } else {
          const float E = (Qv > Bv) ? (Qv - Bv) : 0.f;
          const int64_t slot = (int64_t)a.Hkv * a.T;
          float ts = 0.f;
          for (int j = 0; j < a.ring_cnt; ++j) ts += a.ring[a.ring_read[j] * slot + pos];
          const float Tv = a.ring_cnt ? ts / (float)a.ring_cnt : 0.f;
          a.ring[a.ring_write * slot + pos] = E;
          a.vec_B[pos] = Bv;
          a.vec_EpT[pos] = ((a.terms & 1u) ? E : 0.f) + ((a.terms & 4u) ? Tv : 0.f);
        }
      }
    }
  }

  if constexpr (MODE == PASS_LSE) {
    // merge the two lane halves (same row, different keys)
    const float mo = __shfl_xor(m_run, 32), lo = __shfl_xor(l_run, 32);
    const float m = fmaxf(m_run, mo);
    float l = 0.f;
    if (m != -INFINITY)
      l = l_run * exp2f((m_run - m) * a.c2) + lo * exp2f((mo - m) * a.c2);
    const int r = wave * 32 + l32;
    if (half == 0) {
      a.partials[((int64_t)h * st.total_chunks + gchunk) * a.Rpad + r] =
          make_float2(m == -INFINITY ? -INFINITY : m * a.c2, l);
    }
    // last workgroup of this (sequence, KV head) merges all chunk partials
    __threadfence();
    __syncthreads();
    __shared__ int s_last;
    if (t == 0) {
      const unsigned nch = (unsigned)(st.chunk_base[b + 1] - st.chunk_base[b]);
      const unsigned old = __hip_atomic_fetch_add(&a.counters[b * a.Hkv + h], 1u,
                                                  __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (old == nch - 1) ? 1 : 0;
    }
    __syncthreads();
    if (s_last) {
      __threadfence();
      const int nch = st.chunk_base[b + 1] - st.chunk_base[b];
      const float2 *pp = a.partials + ((int64_t)h * st.total_chunks + st.chunk_base[b]) * a.Rpad;
      for (int row = t; row < a.Rpad; row += nt) {
        float mm = -INFINITY;
        for (int cc = 0; cc < nch; ++cc) mm = fmaxf(mm, pp[(int64_t)cc * a.Rpad + row].x);
        float ll = 0.f;
        if (mm != -INFINITY) {
          for (int cc = 0; cc < nch; ++cc) {
            const float2 v = pp[(int64_t)cc * a.Rpad + row];
            if (v.x != -INFINITY) ll += v.y * exp2f(v.x - mm);
          }
        }
        const float lse2 = (row < a.R) ? mm + log2f(ll) : INFINITY;
        a.lse2[((int64_t)b * a.Hkv + h) * a.Rpad + row] = lse2;
        if (a.lse_user && row < a.R) {
          const int g = row / W, w = row - g * W;
          a.lse_user[((int64_t)b * a.Hq + (int64_t)h * a.G + g) * W + w] = lse2 * kLn2;
        }
      }
      if (t == 0) a.counters[b * a.Hkv + h] = 0u;
    }
  }
}

PassGeom pass_geom(int mode, bool bf16, int head_dim, int rpad) {
  PassGeom g;
  g.nw = rpad / 32;
  g.tk = stage_keys(g.nw);
  const int stride = head_dim * (bf16 ? 2 : 4) + 16;
  g.lds = 2 * g.tk * stride;
  if (mode != PASS_LSE) g.lds += 2 * 2 * g.nw * g.tk * (int)sizeof(float);
  return g;
}

// Dynamic LDS above 64 KiB has to be allowed per kernel before launch.
template <typename Kern>
static void allow_lds(Kern kernel, size_t bytes) {
  static size_t granted = 0;
  if (bytes > 64 * 1024 && bytes > granted) {
    hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    granted = bytes;
  }
}

template <int MODE, bool BF16, int D, bool W32>
static hipError_t launch_pass_t(const PassArgs &a, const SeqTable &st, hipStream_t s) {
  const PassGeom g = pass_geom(MODE, BF16, D, a.Rpad);
  dim3 grid(st.total_chunks, a.Hkv), block(64 * g.nw);
  allow_lds(k_pass<MODE, BF16, D, W32>, g.lds);
  hipLaunchKernelGGL((k_pass<MODE, BF16, D, W32>), grid, block, g.lds, s, a, st);
  return hipGetLastError();
}

template <int MODE>
static hipError_t launch_pass_m(bool bf16, int d, bool w32, const PassArgs &a, const SeqTable &st,
                                hipStream_t s) {
  if (bf16) {
    if (d == 128) return w32 ? launch_pass_t<MODE, true, 128, true>(a, st, s)
                             : launch_pass_t<MODE, true, 128, false>(a, st, s);
    return w32 ? launch_pass_t<MODE, true, 64, true>(a, st, s)
               : launch_pass_t<MODE, true, 64, false>(a, st, s);
  }
  if (d == 128) return w32 ? launch_pass_t<MODE, false, 128, true>(a, st, s)
                           : launch_pass_t<MODE, false, 128, false>(a, st, s);
  return w32 ? launch_pass_t<MODE, false, 64, true>(a, st, s)
             : launch_pass_t<MODE, false, 64, false>(a, st, s);
}

hipError_t launch_pass(int mode, bool bf16, int head_dim, bool w32, const PassArgs &a,
                       const SeqTable &st, hipStream_t s) {
  if (mode == PASS_LSE) return launch_pass_m<PASS_LSE>(bf16, head_dim, false, a, st, s);
  if (mode == PASS_SCORE) return launch_pass_m<PASS_SCORE>(bf16, head_dim, w32, a, st, s);
  return launch_pass_m<PASS_FUSED>(bf16, head_dim, w32, a, st, s);
}

// ---------------------------------------------------------------- block helpers
struct SelShared {
  unsigned hist[kHistBins];
  unsigned red_u[kSelThreads / 64];
  double red_d[4][kSelThreads / 64];
  unsigned bc_u[4];
  double bc_d[4];
  int bc_i[4];
};

__device__ __forceinline__ unsigned wave_min_u(unsigned v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = min(v, (unsigned)__shfl_xor((int)v, o));
  return v;
}
__device__ __forceinline__ unsigned wave_max_u(unsigned v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = max(v, (unsigned)__shfl_xor((int)v, o));
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ unsigned block_min_u(unsigned v, SelShared &ss) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  v = wave_min_u(v);
  if (lane == 0) ss.red_u[wave] = v;
  __syncthreads();
  if (wave == 0) {
    unsigned x = (lane < kSelThreads / 64) ? ss.red_u[lane] : 0xffffffffu;
    x = wave_min_u(x);
    if (lane == 0) ss.bc_u[0] = x;
  }
  __syncthreads();
  return ss.bc_u[0];
}
__device__ unsigned block_max_u(unsigned v, SelShared &ss) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  v = wave_max_u(v);
  if (lane == 0) ss.red_u[wave] = v;
  __syncthreads();
  if (wave == 0) {
    unsigned x = (lane < kSelThreads / 64) ? ss.red_u[lane] : 0u;
    x = wave_max_u(x);
    if (lane == 0) ss.bc_u[1] = x;
  }
  __syncthreads();
  return ss.bc_u[1];
}
// Sum of four doubles over the block; result in out[0..3] for every thread.
__device__ void block_sum4_d(double v0, double v1, double v2, double v3, SelShared &ss, double *out) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  v0 = wave_sum_d(v0); v1 = wave_sum_d(v1); v2 = wave_sum_d(v2); v3 = wave_sum_d(v3);
  if (lane == 0) { ss.red_d[0][wave] = v0; ss.red_d[1][wave] = v1; ss.red_d[2][wave] = v2; ss.red_d[3][wave] = v3; }
  __syncthreads();
  if (t < 4) {
    double s = 0.0;
    for (int w = 0; w < kSelThreads / 64; ++w) s += ss.red_d[t][w];   // fixed order
    ss.bc_d[t] = s;
  }
  __syncthreads();
  out[0] = ss.bc_d[0]; out[1] = ss.bc_d[1]; out[2] = ss.bc_d[2]; out[3] = ss.bc_d[3];
  __syncthreads();
}
// Exclusive prefix sum over threads in index order.
__device__ unsigned block_excl_scan_u(unsigned v, SelShared &ss) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  unsigned x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned y = (unsigned)__shfl_up((int)x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) ss.red_u[wave] = x;
  __syncthreads();
  unsigned before = 0;
  for (int w = 0; w < wave; ++w) before += ss.red_u[w];
  __syncthreads();
  return before + x - v;
}

// Order-preserving map of a float to uint32 (larger float -> larger key);
// -0 is folded to +0.  0 is reserved for "not a candidate".
__device__ __forceinline__ unsigned float_key(float x) {
  x = x + 0.0f;
  const unsigned u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// k-th largest key among the block's non-zero keys (1 <= k <= count), by
// MSB-first 11-bit histogram narrowing of the candidate range.  Returns the
// key value xk and need = k - #{keys > xk} (how many ties at xk are taken).
template <int PER>
__device__ void block_select(const unsigned (&key)[PER], int k, unsigned &xk, int &need,
                             SelShared &ss) {
  const int t = threadIdx.x;
  unsigned lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (key[j]) { lo = min(lo, key[j]); hi = max(hi, key[j]); }
  lo = block_min_u(lo, ss);
  hi = block_max_u(hi, ss);
  need = k;
  while (lo != hi) {
    const unsigned range = hi - lo;
    const int sh = max(0, 32 - __clz((int)range) - 11);
    for (int q = t; q < kHistBins; q += kSelThreads) ss.hist[q] = 0u;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const unsigned x = key[j];
      if (x >= lo && x <= hi) atomicAdd(&ss.hist[(x - lo) >> sh], 1u);
    }
    __syncthreads();
    if (t < 64) {
      const int lane = t;
      unsigned cs = 0;
      for (int q = 0; q < 32; ++q) cs += ss.hist[lane * 32 + q];
      // suffix sums over lanes: suf = # in bins of lanes >= lane
      unsigned suf = cs;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const unsigned y = (unsigned)__shfl_down((int)suf, o);
        if (lane + o < 64) suf += y;
      }
      const unsigned above_lane = suf - cs;
      if (above_lane < (unsigned)need && (unsigned)need <= suf) {
        unsigned acc = above_lane;
        int bs = lane * 32;
        for (int q = 31; q >= 0; --q) {
          const unsigned hq = ss.hist[lane * 32 + q];
          if (acc + hq >= (unsigned)need) { bs = lane * 32 + q; break; }
          acc += hq;
        }
        ss.bc_i[0] = bs;
        ss.bc_i[1] = (int)acc;
      }
    }
    __syncthreads();
    const int bs = ss.bc_i[0];
    need -= ss.bc_i[1];
    const unsigned nlo = lo + ((unsigned)bs << sh);
    const unsigned span = (sh >= 32) ? 0xffffffffu : ((1u << sh) - 1u);
    const unsigned nhi = (hi - nlo <= span) ? hi : nlo + span;
    lo = nlo;
    hi = nhi;
    __syncthreads();
  }
  xk = lo;
}

// ---------------------------------------------------------------- select kernel
template <int PER, int MODE>
__global__ __launch_bounds__(kSelThreads) void k_select(SelArgs a, SeqTable st) {
  extern __shared__ __align__(16) float arr[];     // [n] E, then V, then S, then slot table
  __shared__ SelShared ss;
  const int b = blockIdx.x, h = blockIdx.y, t = threadIdx.x;
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;                           // candidate set [0, nc)
  const int K = st.budget[b];
  const int64_t base = (int64_t)h * a.T + st.cu[b];
  const int i0 = t * PER;

  float Bv[PER], Vv[PER];
  float lam = 0.f;

  if constexpr (MODE != SEL_TOPK) {
    // E of this layer into LDS; own B and E+T into registers.
    for (int i = t; i < n; i += kSelThreads) arr[i] = a.ring_E[base + i];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = i0 + j;
      Bv[j] = (i < n) ? a.vec_B[base + i] : 0.f;
      Vv[j] = (i < n) ? a.vec_EpT[base + i] : 0.f;
    }
    __syncthreads();
    // L = P_r E: truncated box mean, sliding sum in double (Eq. intra_layer_coherence)
    if (i0 < n) {
      const int r = a.radius;
      int lo = max(0, i0 - r), hi = min(n - 1, i0 + r);
      double acc = 0.0;
      for (int u = lo; u <= hi; ++u) acc += (double)arr[u];
      const double inv_full = 1.0 / (double)(2 * r + 1);
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int i = i0 + j;
        if (i < n) {
          const int cnt = hi - lo + 1;
          const double L = acc * ((cnt == 2 * r + 1) ? inv_full : 1.0 / (double)cnt);
          if (a.terms & 2u) Vv[j] += (float)(L > 0.0 ? L : 0.0);
          if constexpr (MODE == SEL_CALIB) {
            if (a.out_E) a.out_E[base + i] = arr[i];
          }
          // slide the window to i+1
          if (i + 1 + r <= n - 1) acc += (double)arr[i + 1 + r];
          if (i - r >= 0) acc -= (double)arr[i - r];
          lo = max(0, i + 1 - r);
          hi = min(n - 1, i + 1 + r);
        }
      }
    }

    // Scale-matching set: top M = min(rho K, |I|) of B over I (Eq. scale_matching_set).
    int M = (int)floorf(a.rho * (float)K);
    if (M > nc) M = nc;
    if (M < 0) M = 0;
    double sums[4] = {0.0, 0.0, 0.0, 0.0};
    unsigned xm = 0;
    if (M > 0 && a.use_last_query) {
      unsigned key[PER];
#pragma unroll
      for (int j = 0; j < PER; ++j) key[j] = (i0 + j < nc) ? float_key(Bv[j]) : 0u;
      int need = 0;
      block_select<PER>(key, M, xm, need, ss);
      unsigned eq_own = 0;
#pragma unroll
      for (int j = 0; j < PER; ++j) eq_own += (key[j] == xm) ? 1u : 0u;
      unsigned e = block_excl_scan_u(eq_own, ss);
      // moments of B (shifted by the M-th value) and V over the set, in double
      const float bref = __uint_as_float(xm & 0x80000000u ? (xm & 0x7fffffffu) : ~xm);
      double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        bool sel = false;
        if (key[j] > xm) sel = true;
        else if (key[j] == xm) { sel = e < (unsigned)need; ++e; }
        if (sel) {
          const double db = (double)Bv[j] - (double)bref, dv = (double)Vv[j];
          s0 += db; s1 += db * db; s2 += dv; s3 += dv * dv;
        }
      }
      block_sum4_d(s0, s1, s2, s3, ss, sums);
      const double mb = sums[0] / M, mv = sums[2] / M;
      double vb = sums[1] / M - mb * mb, vv = sums[3] / M - mv * mv;
      vb = vb > 0.0 ? vb : 0.0;
      vv = vv > 0.0 ? vv : 0.0;
      const double sb = sqrt(vb), sv = sqrt(vv);
      lam = (float)((double)a.gamma * sb / (sv + (double)a.eps));   // Eq. lambda_solution
    }
    if (t == 0) {
      a.lambda_ws[b * a.Hkv + h] = lam;
      if (a.out_lambda) a.out_lambda[b * a.Hkv + h] = lam;
    }
    __syncthreads();   // all reads of E in LDS are done

    // S = B + lambda V (Eq. bacon_score)
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = i0 + j;
      if (i < n) {
        const float S = fmaf(lam, Vv[j], Bv[j]);
        if constexpr (MODE == SEL_CALIB) {
          a.out_S[base + i] = S;
          if (a.out_V) a.out_V[base + i] = Vv[j];
        } else {
          arr[i] = S;
        }
      }
    }
    if constexpr (MODE == SEL_CALIB) return;
  } else {
    for (int i = t; i < nc; i += kSelThreads) arr[i] = a.in_S[base + i];
  }
  __syncthreads();

  // Pooled score over I and its keys.
  unsigned key[PER];
  {
    const int hp = a.pool_half;
    if (i0 < nc) {
      int lo = max(0, i0 - hp), hi = min(nc - 1, i0 + hp);
      double acc = 0.0;
      for (int u = lo; u <= hi; ++u) acc += (double)arr[u];
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int i = i0 + j;
        key[j] = 0u;
        if (i < nc) {
          const double P = acc / (double)(hi - lo + 1);
          key[j] = float_key((float)P);
          if (i + 1 + hp <= nc - 1) acc += (double)arr[i + 1 + hp];
          if (i - hp >= 0) acc -= (double)arr[i - hp];
          lo = max(0, i + 1 - hp);
          hi = min(nc - 1, i + 1 + hp);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < PER; ++j) key[j] = 0u;
    }
  }
  __syncthreads();   // pooled values read; arr is reused as the slot table

  // Top-K over I (Eq. topk_selection), emitted in ascending position.
  const int kept = min(K, nc);
  int32_t *idx = a.idx + (int64_t)st.idx_base[b] * a.Hkv + (int64_t)h * K;
  int *tbl = reinterpret_cast<int *>(arr);
  if (kept == nc) {
    for (int i = t; i < nc; i += kSelThreads) { idx[i] = i; tbl[i] = i; }
  } else if (kept > 0) {
    unsigned xk = 0;
    int need = 0;
    block_select<PER>(key, kept, xk, need, ss);
    unsigned gt_own = 0, eq_own = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) { gt_own += key[j] > xk; eq_own += key[j] == xk; }
    const unsigned packed = block_excl_scan_u((gt_own << 16) | eq_own, ss);
    unsigned g = packed >> 16, e = packed & 0xffffu;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      int slot = -1;
      if (key[j] > xk) { slot = (int)(g + min(e, (unsigned)need)); ++g; }
      else if (key[j] == xk) { if (e < (unsigned)need) slot = (int)(g + e); ++e; }
      if (slot >= 0) { idx[slot] = i0 + j; tbl[slot] = i0 + j; }
    }
  }
  for (int j = kept + t; j < K; j += kSelThreads) idx[j] = -1;

  if constexpr (MODE == SEL_FUSED) {
    if (!a.do_gather) return;
    for (int w = t; w < a.W; w += kSelThreads) tbl[kept + w] = nc + w;
    __syncthreads();
    const int pieces = a.row_bytes / 16;
    const int rows = K + a.W;
    const int total = rows * pieces;
    const unsigned char *ks = static_cast<const unsigned char *>(a.k);
    const unsigned char *vs = static_cast<const unsigned char *>(a.v);
    unsigned char *ko = static_cast<unsigned char *>(a.k_out);
    unsigned char *vo = static_cast<unsigned char *>(a.v_out);
    const int64_t rs = (int64_t)a.Hkv * a.row_bytes;
    for (int q = t; q < total; q += kSelThreads) {
      const int r = q / pieces, p = q - r * pieces;
      const int src = (r < kept + a.W) ? tbl[r] : -1;
      const int64_t dst = ((int64_t)(st.kept_base[b] + r) * a.Hkv + h) * a.row_bytes + 16 * p;
      u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = u32x4{0u, 0u, 0u, 0u};
      if (src >= 0) {
        const int64_t so = ((int64_t)(st.cu[b] + src) * a.Hkv + h) * a.row_bytes + 16 * p;
        kv = *reinterpret_cast<const u32x4 *>(ks + so);
        vv = *reinterpret_cast<const u32x4 *>(vs + so);
      }
      *reinterpret_cast<u32x4 *>(ko + dst) = kv;
      *reinterpret_cast<u32x4 *>(vo + dst) = vv;
      (void)rs;
    }
  }
}

template <int PER>
static hipError_t launch_select_p(int mode, int max_len, const SelArgs &a, const SeqTable &st,
                                  hipStream_t s) {
  dim3 grid(st.batch, a.Hkv), block(kSelThreads);
  const size_t lds = (size_t)max_len * sizeof(float);
  if (mode == SEL_FUSED) {
    allow_lds(k_select<PER, SEL_FUSED>, lds);
    hipLaunchKernelGGL((k_select<PER, SEL_FUSED>), grid, block, lds, s, a, st);
  } else if (mode == SEL_CALIB) {
    allow_lds(k_select<PER, SEL_CALIB>, lds);
    hipLaunchKernelGGL((k_select<PER, SEL_CALIB>), grid, block, lds, s, a, st);
  } else {
    allow_lds(k_select<PER, SEL_TOPK>, lds);
    hipLaunchKernelGGL((k_select<PER, SEL_TOPK>), grid, block, lds, s, a, st);
  }
  return hipGetLastError();
}

hipError_t launch_select(int mode, int max_len, const SelArgs &a, const SeqTable &st,
                         hipStream_t s) {
  if (max_len <= 16 * kSelThreads) return launch_select_p<16>(mode, max_len, a, st, s);
  if (max_len <= 32 * kSelThreads) return launch_select_p<32>(mode, max_len, a, st, s);
  return launch_select_p<64>(mode, max_len, a, st, s);
}

// ---------------------------------------------------------------- split calibrate
__global__ __launch_bounds__(256) void k_elem(ElemArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int h = blockIdx.y;
  if (i >= a.T) return;
  const int64_t pos = (int64_t)h * a.T + i;
  const float Bv = a.in_B[pos], Qv = a.in_Q[pos];
  const float E = (Qv > Bv) ? (Qv - Bv) : 0.f;
  const int64_t slot = (int64_t)a.Hkv * a.T;
  float ts = 0.f;
  for (int j = 0; j < a.ring_cnt; ++j) ts += a.ring[a.ring_read[j] * slot + pos];
  const float Tv = a.ring_cnt ? ts / (float)a.ring_cnt : 0.f;
  a.ring[a.ring_write * slot + pos] = E;
  a.vec_B[pos] = Bv;
  a.vec_EpT[pos] = ((a.terms & 1u) ? E : 0.f) + ((a.terms & 4u) ? Tv : 0.f);
}

hipError_t launch_elem(const ElemArgs &a, hipStream_t s) {
  dim3 grid((unsigned)((a.T + 255) / 256), a.Hkv), block(256);
  hipLaunchKernelGGL(k_elem, grid, block, 0, s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- compaction
__global__ __launch_bounds__(256) void k_compact(CompactArgs a, SeqTable st) {
  const int b = blockIdx.x, h = blockIdx.y;
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int K = st.budget[b];
  const int kept = min(K, nc);
  const int32_t *idx = a.idx + (int64_t)st.idx_base[b] * a.Hkv + (int64_t)h * K;
  const int pieces = a.row_bytes / 16;
  const int total = (K + a.W) * pieces;
  const unsigned char *ks = static_cast<const unsigned char *>(a.k);
  const unsigned char *vs = static_cast<const unsigned char *>(a.v);
  unsigned char *ko = static_cast<unsigned char *>(a.k_out);
  unsigned char *vo = static_cast<unsigned char *>(a.v_out);
  for (int q = blockIdx.z * blockDim.x + threadIdx.x; q < total; q += gridDim.z * blockDim.x) {
    const int r = q / pieces, p = q - r * pieces;
    int src = -1;
    if (r < kept) {
      src = idx[r];
      if (src < 0 || src >= n) src = -1;
    } else if (r < kept + a.W) {
      src = nc + (r - kept);
    }
    const int64_t dst = ((int64_t)(st.kept_base[b] + r) * a.Hkv + h) * a.row_bytes + 16 * p;
    u32x4 kv = u32x4{0u, 0u, 0u, 0u}, vv = u32x4{0u, 0u, 0u, 0u};
    if (src >= 0) {
      const int64_t so = ((int64_t)(st.cu[b] + src) * a.Hkv + h) * a.row_bytes + 16 * p;
      kv = *reinterpret_cast<const u32x4 *>(ks + so);
      vv = *reinterpret_cast<const u32x4 *>(vs + so);
    }
    *reinterpret_cast<u32x4 *>(ko + dst) = kv;
    *reinterpret_cast<u32x4 *>(vo + dst) = vv;
  }
}

hipError_t launch_compact(const CompactArgs &a, const SeqTable &st, hipStream_t s) {
  dim3 grid(st.batch, a.Hkv, 4), block(256);
  hipLaunchKernelGGL(k_compact, grid, block, 0, s, a, st);
  return hipGetLastError();
}

__global__ void k_clear_u32(unsigned *p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

hipError_t launch_clear_u32(unsigned *p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_clear_u32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace bacon
