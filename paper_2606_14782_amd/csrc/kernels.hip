// gfx950 kernels of the BACON prefill KV-compression pass.
//
// Pass 1 (PASS_LSE) and pass 2 (PASS_SCORE / PASS_FUSED) each stream the
// layer's keys once.  A workgroup owns one (KV head, key chunk); its waves own
// the 32-row tiles of the G*W window queries of that KV head.  Key stages go
// straight from HBM to LDS (16-byte direct loads) and are consumed by 32x32
// MFMA (bf16: v_mfma_f32_32x32x16_bf16, fp32: v_mfma_f32_32x32x2_f32).
//
//  * Pass 1 computes D = K Q^T so each lane holds one query row: the running
//    row max and sum of exp2 stay in-lane; each chunk writes one (max, sum)
//    partial per row, and a merge kernel forms the row normalisers.
//  * Pass 2 computes D = Q K^T so each lane holds one key: the window mean B
//    and the last-query score Q are in-lane sums over the lane's rows,
//    reduced across row tiles through LDS in a fixed order (deterministic).
//    The fused variant forms E = [Q-B]_+ (Eq. boundary_residual), T from the
//    E history (Eq. inter_layer_persistence), appends E to the history, and
//    adds the B keys of its candidates to the B histogram of the select; the
//    select's calibration kernel forms L = P_r E (Eq. intra_layer_coherence)
//    from the history.
//
// The fused pass then selects in four kernels over segments of kSegLen
// positions, exchanging histograms and short per-segment lists (see the
// "histogram select" section): calibration (V, pooling, the candidates of
// the scale-matching set), score (lambda and the pooled score), candidates of
// the top-K, and the final top-K with the gather of the compacted cache.
// One workgroup per (sequence, KV head) runs the same steps over the whole
// sequence for the split calls.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <math.h>
#include <stdint.h>

#include "internal.h"

namespace bacon {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void g_void;

// s_waitcnt immediate (gfx9 encoding) waiting for vmcnt = 0 only:
// vmcnt bits [3:0] and [15:14] zero, expcnt [6:4] and lgkmcnt [11:8] at max.
constexpr int kWaitVm0 = 0x0F70;
// ... and for lgkmcnt = 0 only (vmcnt at its maximum 63, expcnt at max).
constexpr int kWaitLgkm0 = 0xC07F;

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.44269504088896341f;

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

// The value of lane l ^ 32 (the other half of the wave), through a VALU lane
// swap rather than an LDS permute.
__device__ __forceinline__ float xor32(float v, int half) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(half ? r[0] : r[1]);
}

// Sum over the wave's 64 lanes through DPP moves (pairs, quads, half rows,
// rows) and four lane reads: the same order, and so the same value, in every
// lane.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);    // quad_perm(1, 0, 3, 2)
  v += dpp_f<0x4E>(v);    // quad_perm(2, 3, 0, 1)
  v += dpp_f<0x141>(v);   // row_half_mirror
  v += dpp_f<0x140>(v);   // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}

// Sums over the wave's 64 lanes of eight values at once: lane swaps 32 and
// 16 apart and a DPP exchange 8 apart each halve the values a lane carries
// (keeping the ones its lane group ends with), then three DPP steps sum
// within groups of 8 lanes, where value k ends (lanes 8k..8k+7).  Each sum
// is formed in one fixed order.
__device__ __forceinline__ void wave_sum8(const float (&x)[8], float (&s)[8], int lane) {
  const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
  float y[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x[i]), __float_as_uint(x[i + 4]), false, false);
    y[i] = (b5 ? x[i + 4] : x[i]) + __uint_as_float(b5 ? r[0] : r[1]);
  }
  float z[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(y[i]), __float_as_uint(y[i + 2]), false, false);
    z[i] = (b4 ? y[i + 2] : y[i]) + __uint_as_float(b4 ? r[0] : r[1]);
  }
  float w = (b3 ? z[1] : z[0]) + dpp_f<0x128>(b3 ? z[0] : z[1]);   // row_ror:8
  w += dpp_f<0xB1>(w);
  w += dpp_f<0x4E>(w);
  w += dpp_f<0x141>(w);
#pragma unroll
  for (int k = 0; k < 8; ++k) s[k] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), 8 * k));
}

// Pairwise (tree) sum and max of 16 values: depth 4 instead of a 16-long chain.
__device__ __forceinline__ float tree_sum16(const float *x) {
  const float a0 = (x[0] + x[1]) + (x[2] + x[3]), a1 = (x[4] + x[5]) + (x[6] + x[7]);
  const float a2 = (x[8] + x[9]) + (x[10] + x[11]), a3 = (x[12] + x[13]) + (x[14] + x[15]);
  return (a0 + a1) + (a2 + a3);
}
__device__ __forceinline__ float tree_min16(const float *x) {
  const float a0 = fminf(fminf(x[0], x[1]), fminf(x[2], x[3]));
  const float a1 = fminf(fminf(x[4], x[5]), fminf(x[6], x[7]));
  const float a2 = fminf(fminf(x[8], x[9]), fminf(x[10], x[11]));
  const float a3 = fminf(fminf(x[12], x[13]), fminf(x[14], x[15]));
  return fminf(fminf(a0, a1), fminf(a2, a3));
}
__device__ __forceinline__ float tree_max16(const float *x) {
  const float a0 = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
  const float a1 = fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7]));
  const float a2 = fmaxf(fmaxf(x[8], x[9]), fmaxf(x[10], x[11]));
  const float a3 = fmaxf(fmaxf(x[12], x[13]), fmaxf(x[14], x[15]));
  return fmaxf(fmaxf(a0, a1), fmaxf(a2, a3));
}

// Order-preserving map of a float to uint32 (larger float -> larger key);
// -0 is folded to +0.  0 is reserved for "not a candidate".
__device__ __forceinline__ unsigned float_key(float x) {
  x = x + 0.0f;
  const unsigned u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Bin of a key in the select histograms: bits 30..18 of a non-negative float
// (32 bins per octave); keys of negative values, which the method does not
// produce, share bin 0, so the bins stay monotone in the key.
__device__ __forceinline__ int hbin(unsigned key) {
  return key >= 0x80000000u ? (int)((key >> 18) & (unsigned)(kHBins - 1)) : 0;
}

// A copy of v the compiler cannot see through: stops it from hoisting address
// arithmetic of one phase and keeping it live through the next.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// The value as produced at this point of the program: uses of it wait for
// its loads here, and no later arithmetic moves above.
__device__ __forceinline__ void pin(u32x4 &v) {
  unsigned x = v.x, y = v.y, z = v.z, w = v.w;
  asm volatile("" : "+v"(x), "+v"(y), "+v"(z), "+v"(w));
  v = u32x4{x, y, z, w};
}
__device__ __forceinline__ void pin(float4 &v) {
  float x = v.x, y = v.y, z = v.z, w = v.w;
  asm volatile("" : "+v"(x), "+v"(y), "+v"(z), "+v"(w));
  v = make_float4(x, y, z, w);
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

// Dynamic LDS above 64 KiB has to be allowed per kernel before launch.
template <typename Kern>
static void allow_lds(Kern kernel, size_t bytes) {
  static size_t granted = 0;
  if (bytes > 64 * 1024 && bytes > granted) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    granted = bytes;
  }
}

// ---------------------------------------------------------------- passes
template <bool BF16, int D>
struct PassCfg {
  static constexpr int ES = BF16 ? 2 : 4;
  static constexpr int ROWB = D * ES;          // bytes per key / query row
  static constexpr int NU = ROWB / 32;         // 16-byte units per lane
  static constexpr int PIECES = ROWB / 16;     // 16-byte pieces per row
  // LDS rows are unpadded; the 16-byte piece p of key k sits in slot
  // p ^ (k & SWM), so the 32 keys one MFMA operand read touches fall on
  // different banks.
  static constexpr int SWM = (PIECES < 16 ? PIECES : 16) - 1;
  static constexpr int MAXL = PIECES / 2;      // max staged loads per thread
};

// LDS map of a pass workgroup (bytes):
//   kbuf  2 * tk * ROWB           double-buffered key stages (swizzled pieces)
//   red   2 * 2 * nw * tk floats  per-stage B/Q partials of each row tile  (pass 2)
//   lse   Rpad floats             row normalisers                          (pass 2)
//   cb    chunk floats            B of the chunk                           (fused)
// After the stages the fused pass reuses kbuf for its B histogram.
int pass_lds_bytes(int mode, bool bf16, int head_dim, int rpad, int chunk) {
  const int nw = rpad / 32, tk = stage_keys(nw);
  int bytes = 2 * tk * head_dim * (bf16 ? 2 : 4);
  if (mode == PASS_FUSED && bytes < 4 * kHBins) bytes = 4 * kHBins;   // room for the B histogram
  if (mode != PASS_LSE) bytes += 16 * nw * tk + 4 * rpad;
  if (mode == PASS_FUSED) bytes += 4 * chunk;
  return bytes;
}

// One workgroup of a streaming pass: chunk gchunk of the sequences' keys of
// KV head h.
template <int MODE, bool BF16, int D, bool W32>
__device__ __forceinline__ void pass_body(const PassArgs &a, const SeqTable &st, int gchunk, int h) {
  using C = PassCfg<BF16, D>;
  extern __shared__ __align__(16) unsigned char smem[];
  const int nw = blockDim.x >> 6;
  const int nt = blockDim.x;
  const int tk = stage_keys(nw);
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63, half = lane >> 5, l32 = lane & 31;
  const int b = find_seq(st, gchunk);
  const int c = gchunk - st.chunk_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int k0 = c * a.chunk;
  const int k1 = min(n, k0 + a.chunk);
  const int W = a.W;
  const int wfirst = n - W;                      // position of window row 0
  const int nstages = (k1 - k0 + tk - 1) / tk;

  unsigned char *kbuf = smem;
  const int kbytes = (MODE == PASS_FUSED) ? max(2 * tk * C::ROWB, 4 * kHBins) : 2 * tk * C::ROWB;
  float *red = reinterpret_cast<float *>(smem + kbytes);               // [2][2][nw][tk]
  float *lse_s = red + 4 * nw * tk;                                    // [Rpad]
  float *cb = lse_s + a.Rpad;                                          // [chunk]

  // Stage loader: direct-to-LDS 16-byte loads (no register staging).  LDS
  // slot s of a stage holds piece (s % PIECES) ^ (key & SWM) of key
  // s / PIECES; load instruction i fills the 64 slots [64 i, 64 i + 64),
  // lane l slot 64 i + l, and wave w issues instructions w, w + nw, ...
  // Loads are unconditional: keys past the chunk are clamped to valid
  // addresses (their data is masked).  The thread's global offsets are the
  // same in every full stage: one uniform base plus them.
  const unsigned char *kb = static_cast<const unsigned char *>(a.k) +
                            ((int64_t)st.cu[b] * a.Hkv + h) * C::ROWB;
  const int64_t kstride = (int64_t)a.Hkv * C::ROWB;
  const int nins = tk * C::PIECES / 64;           // load instructions per stage
  int goff[C::MAXL];
#pragma unroll
  for (int j = 0; j < C::MAXL; ++j) {
    const int sl = min(wave + nw * j, nins - 1) * 64 + lane;
    const int key = sl / C::PIECES, pc = (sl % C::PIECES) ^ (key & C::SWM);
    goff[j] = key * (int)kstride + 16 * pc;
  }
  auto fetch = [&](int s) {
    const int key0 = k0 + s * tk;
    unsigned char *dst = kbuf + (s & 1) * tk * C::ROWB;
    if (key0 + tk <= k1) {
      const unsigned char *base = kb + (int64_t)key0 * kstride;
#pragma unroll
      for (int j = 0; j < C::MAXL; ++j) {
        const int i = wave + nw * j;
        if (i < nins)
          __builtin_amdgcn_global_load_lds((const g_void *)(base + goff[j]), (lds_void *)(dst + i * 1024),
                                           16, 0, 0);
      }
    } else {
#pragma unroll
      for (int j = 0; j < C::MAXL; ++j) {
        const int i = wave + nw * j;
        if (i < nins) {
          const int sl = i * 64 + lane;
          const int kk = sl / C::PIECES, pc = (sl % C::PIECES) ^ (kk & C::SWM);
          const int key = min(key0 + kk, k1 - 1);
          __builtin_amdgcn_global_load_lds((const g_void *)(kb + (int64_t)key * kstride + 16 * pc),
                                           (lds_void *)(dst + i * 1024), 16, 0, 0);
        }
      }
    }
  };
  // the direct loads count in vmcnt: wait for all of them before the barrier
  // that publishes a stage
  auto stage_wait = [] { __builtin_amdgcn_s_waitcnt(kWaitVm0); };

  fetch(0);   // first key stage in flight while the prologue runs

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

  // byte offsets of this lane's operand pieces 2u + half of key l32 of a
  // tile, from the tile's first key row
  int koff[C::NU];
#pragma unroll
  for (int u = 0; u < C::NU; ++u) koff[u] = l32 * C::ROWB + 16 * ((2 * u + half) ^ (l32 & C::SWM));

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
    // row normalisers of this (sequence, KV head): merged from pass 1's
    // per-chunk partials by the merge kernel, or given by the caller as the
    // natural-log normalisers of the window rows [B, Hq, W]
    for (int r = t; r < a.Rpad; r += nt) {
      if (a.lse_in) {
        const int g = r / W, w = r - g * W;
        lse_s[r] = r < a.R ? a.lse_in[((int64_t)b * a.Hq + (int64_t)h * a.G + g) * W + w] * kLog2e
                           : INFINITY;
      } else {
        lse_s[r] = a.lse2[((int64_t)b * a.Hkv + h) * a.Rpad + r];
      }
    }
    __syncthreads();
#pragma unroll
    for (int reg = 0; reg < 16; ++reg) {
      const int r = wave * 32 + acc_row(reg, half);
      nl[reg] = -lse_s[r];
      wrow[reg] = (r < a.R) ? r % W : W;
      if (!W32 && r < a.R && (r % W) == W - 1) lastmask |= 1u << reg;
    }
  }
  stage_wait();
  __syncthreads();
  for (int s = 0; s < nstages; ++s) {
    const int buf = s & 1;
    const int ntile = min(tk, k1 - (k0 + s * tk));
    if (s + 1 < nstages) fetch(s + 1);
    const unsigned char *kl = kbuf + buf * tk * C::ROWB;
    // The tiles of a stage are unrolled (a tile's row offset is a constant in
    // the LDS read instruction) and software-pipelined: the MFMA chain of
    // tile kt + 1 is issued before the vector work on tile kt, so the matrix
    // and vector units overlap inside one wave.
    auto tile_mma = [&](int kt) {
      const unsigned char *kr = kl + kt * 32 * C::ROWB;
      f32x16 acc = {};
#pragma unroll
      for (int u = 0; u < C::NU; ++u) {
        const u32x4 kv = *reinterpret_cast<const u32x4 *>(kr + koff[u]);
        if constexpr (MODE == PASS_LSE) acc = mfma_unit<BF16>(kv, qf[u], acc);   // D = K Q^T
        else acc = mfma_unit<BF16>(qf[u], kv, acc);                              // D = Q K^T
      }
      return acc;
    };
    auto tile_post = [&](int kt, f32x16 acc) {
      const int kbase = k0 + s * tk + kt * 32;   // first key of the tile (sequence-relative)
      if constexpr (MODE == PASS_LSE) {
        // acc[reg]: key kbase + acc_row(reg, half), row = wave*32 + l32
        const bool edge = (kbase + 31 >= k1) || (kbase + 31 > wfirst);
        if (edge) {
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) {
            const int key = kbase + acc_row(reg, half);
            if (!(key < k1 && key <= tpos_row)) acc[reg] = -INFINITY;
          }
        }
        float av[16];
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) av[reg] = acc[reg];
        const float mt = tree_max16(av);
        if (mt > m_run) {
          l_run *= __builtin_amdgcn_exp2f((m_run - mt) * a.c2);
          m_run = mt;
        }
        if (m_run != -INFINITY) {
          const float off = -m_run * a.c2;
          float ev[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) ev[reg] = __builtin_amdgcn_exp2f(fmaf(av[reg], a.c2, off));
          l_run += tree_sum16(ev);
        }
      } else {
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
        float bs = tree_sum16(p), qs = 0.f;
        if constexpr (W32) {
          qs = half ? p[15] : 0.f;
        } else {
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) qs += ((lastmask >> reg) & 1u) ? p[reg] : 0.f;
        }
        bs += xor32(bs, half);
        qs += xor32(qs, half);
        if (half == 0) {
          red[((buf * 2 + 0) * nw + wave) * tk + kt * 32 + l32] = bs;
          red[((buf * 2 + 1) * nw + wave) * tk + kt * 32 + l32] = qs;
        }
      }
    };
    const int ntiles = (ntile + 31) / 32;        // 1..4
    f32x16 cur = tile_mma(0);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      if (kt >= ntiles) break;
      f32x16 nxt = cur;
      if (kt + 1 < ntiles) nxt = tile_mma(kt + 1);
      tile_post(kt, cur);
      cur = nxt;
    }
    stage_wait();
    __syncthreads();
    if constexpr (MODE != PASS_LSE) {
      // Stage epilogue: fixed-order reduction over row tiles, one key per thread.
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
          // E (Eq. boundary_residual) to this layer's history slot; the
          // calibration kernel forms L, T and V from the history
          a.ring[a.ring_write * a.ring_stride + pos] = (Qv > Bv) ? (Qv - Bv) : 0.f;
          a.vec_B[pos] = Bv;
          cb[s * tk + t] = Bv;
        }
      }
    }
  }

  if constexpr (MODE == PASS_FUSED) {
    __syncthreads();
    // B histogram of the chunk's candidates (positions before the window) in
    // the key-stage buffers, added to one of kHCopies copies of the
    // (sequence, KV head) histogram of the select bin by bin (workgroup w
    // takes copy w % kHCopies: consecutive workgroups run on different XCDs,
    // so a hot bin takes few atomics per copy); only the bins between the
    // chunk's smallest and largest are cleared and flushed.
    unsigned *hist = reinterpret_cast<unsigned *>(kbuf);
    const int ncnd = max(0, min(k1, wfirst) - k0);
    int blo = kHBins, bhi = -1;
    for (int p = t; p < ncnd; p += nt) {
      const int q = hbin(float_key(cb[p]));
      blo = min(blo, q);
      bhi = max(bhi, q);
    }
    blo = __reduce_min_sync(~0ull, blo);
    bhi = __reduce_max_sync(~0ull, bhi);
    float *mm = red;                              // wave minima / maxima (red is free here)
    if (lane == 0) { mm[wave] = __int_as_float(blo); mm[16 + wave] = __int_as_float(bhi); }
    __syncthreads();
    blo = kHBins;
    bhi = -1;
    for (int w = 0; w < nw; ++w) {
      blo = min(blo, __float_as_int(mm[w]));
      bhi = max(bhi, __float_as_int(mm[16 + w]));
    }
    for (int q = blo + t; q <= bhi; q += nt) hist[q] = 0u;
    __syncthreads();
    for (int p = t; p < ncnd; p += nt) atomicAdd(&hist[hbin(float_key(cb[p]))], 1u);
    __syncthreads();
    const int copy = (h * st.total_chunks + gchunk) % kHCopies;
    unsigned *gh = a.hist_B + (((int64_t)b * a.Hkv + h) * kHCopies + copy) * kHBins;
    for (int q = blo + t; q <= bhi; q += nt) {
      const unsigned cnt = hist[q];
      if (cnt) atomicAdd(&gh[q], cnt);
    }
  }

  if constexpr (MODE == PASS_LSE) {
    // merge the two lane halves (same row, different keys) and store the partial
    const float mo = xor32(m_run, half), lo = xor32(l_run, half);
    const float m = fmaxf(m_run, mo);
    float l = 0.f;
    if (m != -INFINITY)
      l = l_run * __builtin_amdgcn_exp2f((m_run - m) * a.c2) + lo * __builtin_amdgcn_exp2f((mo - m) * a.c2);
    const int r = wave * 32 + l32;
    if (half == 0) {
      a.partials[((int64_t)h * st.total_chunks + gchunk) * a.Rpad + r] =
          make_float2(m == -INFINITY ? -INFINITY : m * a.c2, l);
    }
  }
}

template <int MODE, bool BF16, int D, bool W32>
__global__ __launch_bounds__(512) void k_pass(PassArgs a, SeqTable st) {
  pass_body<MODE, BF16, D, W32>(a, st, blockIdx.x, blockIdx.y);
}

// Pass 2 of one layer (a2) and pass 1 of the next (a1) in one grid, as the
// key-register k_krdual: the first total_chunks columns take a2.
template <bool BF16, int D, bool W32>
__global__ __launch_bounds__(512) void k_pass_dual(PassArgs a2, PassArgs a1, SeqTable st) {
  if ((int)blockIdx.x < st.total_chunks)
    pass_body<PASS_FUSED, BF16, D, W32>(a2, st, blockIdx.x, blockIdx.y);
  else
    pass_body<PASS_LSE, BF16, D, false>(a1, st, blockIdx.x - st.total_chunks, blockIdx.y);
}

template <bool BF16, int D, bool W32>
static hipError_t launch_pass_dual_t(const PassArgs &a2, const PassArgs &a1, const SeqTable &st,
                                     hipStream_t s) {
  const int nw = a2.Rpad / 32;
  const int lds = std::max(pass_lds_bytes(PASS_FUSED, BF16, D, a2.Rpad, a2.chunk),
                           pass_lds_bytes(PASS_LSE, BF16, D, a1.Rpad, a1.chunk));
  if (lds > kLdsBytes || a1.Rpad != a2.Rpad || a1.chunk != a2.chunk) return hipErrorInvalidValue;
  dim3 grid(2 * st.total_chunks, a2.Hkv), block(64 * nw);
  allow_lds(k_pass_dual<BF16, D, W32>, lds);
  hipLaunchKernelGGL((k_pass_dual<BF16, D, W32>), grid, block, lds, s, a2, a1, st);
  return hipGetLastError();
}

hipError_t launch_pass_dual(bool bf16, int d, bool w32, const PassArgs &a2, const PassArgs &a1,
                            const SeqTable &st, hipStream_t s) {
  if (bf16) {
    if (d == 128) return w32 ? launch_pass_dual_t<true, 128, true>(a2, a1, st, s)
                             : launch_pass_dual_t<true, 128, false>(a2, a1, st, s);
    return w32 ? launch_pass_dual_t<true, 64, true>(a2, a1, st, s)
               : launch_pass_dual_t<true, 64, false>(a2, a1, st, s);
  }
  if (d == 128) return w32 ? launch_pass_dual_t<false, 128, true>(a2, a1, st, s)
                           : launch_pass_dual_t<false, 128, false>(a2, a1, st, s);
  return w32 ? launch_pass_dual_t<false, 64, true>(a2, a1, st, s)
             : launch_pass_dual_t<false, 64, false>(a2, a1, st, s);
}

template <int MODE, bool BF16, int D, bool W32>
static hipError_t launch_pass_t(const PassArgs &a, const SeqTable &st, hipStream_t s) {
  const int nw = a.Rpad / 32;
  const int lds = pass_lds_bytes(MODE, BF16, D, a.Rpad, a.chunk);
  if (lds > kLdsBytes) return hipErrorInvalidValue;
  dim3 grid(st.total_chunks, a.Hkv), block(64 * nw);
  allow_lds(k_pass<MODE, BF16, D, W32>, lds);
  hipLaunchKernelGGL((k_pass<MODE, BF16, D, W32>), grid, block, lds, s, a, st);
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

// Row normalisers of each (sequence, KV head) from the per-chunk (max, sum)
// partials of pass 1.  A workgroup takes 16 rows: thread t merges row t % 16
// over the chunks congruent to t / 16 (mod 16), kMergeBatch loads in flight
// per batch; the 16 parts of a row are combined through LDS in a fixed order.
constexpr int kMergeRows = 16, kMergeParts = 16, kMergeBatch = 8;
constexpr int kMergeThreads = kMergeRows * kMergeParts;
// Row group rg of (sequence b, KV head h) by the kMergeThreads threads t of
// one group; `valid` false: the group only takes part in the barrier.
__device__ __forceinline__ void merge_rows(const PassArgs &a, const SeqTable &st, int rg, int b,
                                           int h, int t, float2 (*mrg)[kMergeRows], bool valid) {
  const int row = rg * kMergeRows + (t % kMergeRows), part = t / kMergeRows;
  const int nch = valid ? st.chunk_base[b + 1] - st.chunk_base[b] : 0;
  const float2 *pp = a.partials + ((int64_t)h * st.total_chunks + st.chunk_base[b]) * a.Rpad + row;
  float mm = -INFINITY, ll = 0.f;
  for (int c0 = part; c0 < nch; c0 += kMergeParts * kMergeBatch) {
    float2 v[kMergeBatch];
#pragma unroll
    for (int j = 0; j < kMergeBatch; ++j) v[j] = pp[(int64_t)min(c0 + kMergeParts * j, nch - 1) * a.Rpad];
#pragma unroll
    for (int j = 0; j < kMergeBatch; ++j)
      if (c0 + kMergeParts * j >= nch) v[j] = make_float2(-INFINITY, 0.f);
    float mb = mm;
#pragma unroll
    for (int j = 0; j < kMergeBatch; ++j) mb = fmaxf(mb, v[j].x);
    if (mb != -INFINITY) {
      float acc = (mm == -INFINITY) ? 0.f : ll * __builtin_amdgcn_exp2f(mm - mb);
#pragma unroll
      for (int j = 0; j < kMergeBatch; ++j)
        if (v[j].x != -INFINITY) acc += v[j].y * __builtin_amdgcn_exp2f(v[j].x - mb);
      ll = acc;
      mm = mb;
    }
  }
  mrg[part][t % kMergeRows] = make_float2(mm, ll);
  __syncthreads();
  if (valid && t < kMergeRows) {
    float mx = -INFINITY;
    for (int q = 0; q < kMergeParts; ++q) mx = fmaxf(mx, mrg[q][t].x);
    float sx = 0.f;
    if (mx != -INFINITY)
      for (int q = 0; q < kMergeParts; ++q) {
        const float2 pq = mrg[q][t];
        if (pq.x != -INFINITY) sx += pq.y * __builtin_amdgcn_exp2f(pq.x - mx);
      }
    const float lse2 = (row < a.R) ? mx + log2f(sx) : INFINITY;
    a.lse2[((int64_t)b * a.Hkv + h) * a.Rpad + row] = lse2;
    if (a.lse_user && row < a.R) {
      const int W = a.W, g = row / W, w = row - g * W;
      a.lse_user[((int64_t)b * a.Hq + (int64_t)h * a.G + g) * W + w] = lse2 * kLn2;
    }
  }
}

__global__ __launch_bounds__(kMergeThreads) void k_lse_merge(PassArgs a, SeqTable st) {
  __shared__ float2 mrg[kMergeParts][kMergeRows];
  merge_rows(a, st, blockIdx.x, blockIdx.y, blockIdx.z, threadIdx.x, mrg, true);
}

hipError_t launch_lse_merge(const PassArgs &a, const SeqTable &st, hipStream_t s) {
  if (a.Rpad % kMergeRows) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_lse_merge, dim3(a.Rpad / kMergeRows, st.batch, a.Hkv),
                     dim3(kMergeThreads), 0, s, a, st);
  return hipGetLastError();
}

hipError_t launch_pass(int mode, bool bf16, int head_dim, bool w32, const PassArgs &a,
                       const SeqTable &st, hipStream_t s) {
  if (mode == PASS_LSE) return launch_pass_m<PASS_LSE>(bf16, head_dim, false, a, st, s);
  if (mode == PASS_SCORE) return launch_pass_m<PASS_SCORE>(bf16, head_dim, w32, a, st, s);
  return launch_pass_m<PASS_FUSED>(bf16, head_dim, w32, a, st, s);
}

// ---------------------------------------------------------------- key-register passes
// The two K passes for bf16 keys with up to 128 window rows, in a second
// design: waves own keys instead of query rows.  A workgroup of kKrWaves
// waves takes the chunk of kr_keys() keys of one KV head; each wave loads its
// KT key tiles straight into registers, in the MFMA operand layout (lane l:
// key l % 32, the 16-byte units of the k-slice l / 32), which is the A operand
// of pass 1 (D = K Q^T) and the B operand of pass 2 (D = Q K^T).  The window
// queries sit in LDS, swizzled like the key stages.  A wave's key loads are
// all in flight at once and each tile is worked on as soon as it has landed;
// pass 2 sums B and Q over the rows inside the wave, so the tiles need no
// workgroup barrier.  Pass 1 writes per-chunk (max, sum) partials that the
// merge kernel turns into the row normalisers, as in the streaming design.
template <bool BF16, int D>
struct KrCfg {
  static constexpr int NU = PassCfg<BF16, D>::NU;
  static constexpr int KT = 32 / NU < 4 ? 32 / NU : 4;   // key tiles per wave: up to 128 registers of keys
  static constexpr int KPW = kKrWaves * KT * 32;         // keys per workgroup
};

int kr_keys(bool bf16, int head_dim) {
  if (bf16) return head_dim == 128 ? KrCfg<true, 128>::KPW : KrCfg<true, 64>::KPW;
  return head_dim == 128 ? KrCfg<false, 128>::KPW : KrCfg<false, 64>::KPW;
}

// Row tiles a workgroup holds for Rpad window rows (0: not covered).
static int kr_row_tiles(int rpad) { return rpad <= 64 ? 2 : (rpad <= 128 ? 4 : 0); }

// LDS map of a key-register workgroup (bytes), NR = 32 * row tiles:
//   qbuf  max(NR * ROWB, 4 * kHBins)        window queries; the B histogram after pass 2
//   part  kKrWaves * NR float2              per-wave row partials (pass 1)
//   nlc   NR floats                         -lse / c2 of each row (pass 2)
//   cb    KPW floats                        B of the chunk's keys (fused)
int kr_lds_bytes(bool bf16, int head_dim, int rpad) {
  const int nr = 32 * kr_row_tiles(rpad), rowb = head_dim * (bf16 ? 2 : 4), kpw = kr_keys(bf16, head_dim);
  return std::max(nr * rowb, 4 * kHBins) + 8 * kKrWaves * nr + 4 * nr + 4 * kpw;
}

// One workgroup of a key-register pass: chunk gchunk of the sequences' keys
// of KV head h.
template <int MODE, int D, bool W32, int NRT>
__device__ __forceinline__ void krpass_body(const PassArgs &a, const SeqTable &st, int gchunk, int h) {
  using C = PassCfg<true, D>;
  constexpr int NU = C::NU, KT = KrCfg<true, D>::KT, KPW = KrCfg<true, D>::KPW;
  constexpr int NT = 64 * kKrWaves, NR = 32 * NRT;
  constexpr bool FUSED = MODE == PASS_FUSED;
  extern __shared__ __align__(16) unsigned char smem[];
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63, half = lane >> 5, l32 = lane & 31;
  const int b = find_seq(st, gchunk);
  const int c = gchunk - st.chunk_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int k0 = c * KPW, k1 = min(n, k0 + KPW);
  const int W = a.W, wfirst = n - W;
  const int64_t vrow = (int64_t)h * a.T + st.cu[b];      // [Hkv, T] index of the sequence's position 0

  unsigned char *qbuf = smem;
  float2 *part = reinterpret_cast<float2 *>(smem + max(NR * C::ROWB, 4 * kHBins));
  float *nlc = reinterpret_cast<float *>(part + kKrWaves * NR);
  float *cb = nlc + NR;

  // ---- loads, in this order: the window queries, the row normalisers
  // (pass 2), the first key tile; once the first group is in LDS, the other
  // key tiles.  Everything goes through
  // registers, so each use waits only for its own loads.  Query slot s of a
  // row holds piece s ^ (row & SWM); rows past the last real one repeat it
  // (their results are discarded).
  constexpr int QP = NR * C::PIECES / NT;                  // query pieces per thread
  u32x4 qv[QP];
#pragma unroll
  for (int j = 0; j < QP; ++j) {
    const int i = t + j * NT, row = i / C::PIECES, pc = i % C::PIECES;
    const int rr = min(row, a.R - 1), g = rr / W, w = rr - g * W;
    qv[j] = *reinterpret_cast<const u32x4 *>(static_cast<const unsigned char *>(a.q) +
        ((int64_t)(b * W + w) * a.Hq + (int64_t)h * a.G + g) * C::ROWB + 16 * pc);
  }
  float lsev = 0.f;
  if constexpr (FUSED) {
    // row normalisers: merged from pass 1 (log2 units), or the caller's
    // natural-log normalisers of the window rows [B, Hq, W]
    const int r = min(t, a.R - 1), g = r / W, w = r - g * W;
    const float *src = a.lse_in ? a.lse_in + ((int64_t)b * a.Hq + (int64_t)h * a.G + g) * W + w
                                : a.lse2 + ((int64_t)b * a.Hkv + h) * a.Rpad + r;
    lsev = *src;
  }
  const int64_t kstride = (int64_t)a.Hkv * C::ROWB;
  const unsigned char *kb = static_cast<const unsigned char *>(a.k) +
                            ((int64_t)st.cu[b] * a.Hkv + h) * C::ROWB + 16 * half;
  u32x4 kr[KT][NU];
  auto load_tile = [&](int kt) {
    const int key = min(k0 + (wave * KT + kt) * 32 + l32, k1 - 1);
    const unsigned char *kp = kb + (int64_t)key * kstride;
#pragma unroll
    for (int u = 0; u < NU; ++u) kr[kt][u] = *reinterpret_cast<const u32x4 *>(kp + 32 * u);
  };
  asm volatile("" ::: "memory");
  load_tile(0);
  asm volatile("" ::: "memory");
  // the first group is taken here, after the first key tile was issued
#pragma unroll
  for (int j = 0; j < QP; ++j) pin(qv[j]);
  if constexpr (FUSED) {
    asm volatile("" : "+v"(lsev));
    // pad rows (and rows past Rpad) get lse = +inf: probability 0
    if (a.lse_in) lsev *= kLog2e;
    if (t < NR) nlc[t] = t < a.R ? -lsev / a.c2 : -INFINITY;
  }
#pragma unroll
  for (int j = 0; j < QP; ++j) {
    const int i = t + j * NT, row = i / C::PIECES, pc = i % C::PIECES;
    *reinterpret_cast<u32x4 *>(qbuf + row * C::ROWB + 16 * (pc ^ (row & C::SWM))) = qv[j];
  }
  // the LDS writes are visible to the workgroup after the barrier (a bare one:
  // the fence of __syncthreads would also wait for the key tile in flight)
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  asm volatile("" ::: "memory");

  // byte offsets of this lane's operand pieces 2u + half of query row l32 of a
  // row tile, from the tile's first row
  int koff[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) koff[u] = l32 * C::ROWB + 16 * ((2 * u + half) ^ (l32 & C::SWM));
  // key tile kt against the NRT row tiles: each key unit feeds one MFMA chain
  // per row tile.  The query fragments of unit u + 1 are read while the MFMAs
  // of unit u run; scheduling barriers keep the compiler from reading further
  // ahead (the keys take half of the register file).
  auto tiles = [&](int kt, int j0, auto &acc, bool keys_first) {
    constexpr int NJ = sizeof(acc) / sizeof(acc[0]);
    u32x4 qf[2][NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      qf[0][j] = *reinterpret_cast<const u32x4 *>(qbuf + (j0 + j) * 32 * C::ROWB + koff[0]);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      if (u + 1 < NU) {
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          qf[(u + 1) & 1][j] = *reinterpret_cast<const u32x4 *>(qbuf + (j0 + j) * 32 * C::ROWB + koff[u + 1]);
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc[j] = keys_first ? mfma_unit<true>(kr[kt][u], qf[u & 1][j], acc[j])
                            : mfma_unit<true>(qf[u & 1][j], kr[kt][u], acc[j]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if constexpr (MODE == PASS_LSE) {
    // ---- pass 1: per-row running max (raw logits) and sum of exp2 over the
    // wave's keys; tiles away from the sequence end and the window take the
    // unmasked, branch-free update
    float m_run[NRT], l_run[NRT];
#pragma unroll
    for (int j = 0; j < NRT; ++j) { m_run[j] = -INFINITY; l_run[j] = 0.f; }
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 < KT) load_tile(kt + 1);
      f32x16 acc[NRT];
#pragma unroll
      for (int j = 0; j < NRT; ++j) acc[j] = f32x16{};
      tiles(kt, 0, acc, true);
      // acc[j][reg]: key kbase + acc_row(reg, half), row j*32 + l32
      const int kbase = k0 + (wave * KT + kt) * 32;
      if (!((kbase + 31 >= k1) || (kbase + 31 > wfirst))) {
#pragma unroll
        for (int j = 0; j < NRT; ++j) {
          float av[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) av[reg] = acc[j][reg];
          const float mn = fmaxf(m_run[j], tree_max16(av));
          const float off = -mn * a.c2;
          float ev[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) ev[reg] = __builtin_amdgcn_exp2f(fmaf(av[reg], a.c2, off));
          l_run[j] = fmaf(l_run[j], __builtin_amdgcn_exp2f(fmaf(m_run[j], a.c2, off)), tree_sum16(ev));
          m_run[j] = mn;
        }
      } else {
#pragma unroll
        for (int j = 0; j < NRT; ++j) {
          const int r = j * 32 + l32;
          const int tpos = wfirst + (r < a.R ? r % W : W - 1);
          float av[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) {
            const int key = kbase + acc_row(reg, half);
            av[reg] = (key < k1 && key <= tpos) ? acc[j][reg] : -INFINITY;
          }
          const float mn = fmaxf(m_run[j], tree_max16(av));
          const float off = mn == -INFINITY ? 0.f : -mn * a.c2;
          float ev[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) ev[reg] = __builtin_amdgcn_exp2f(fmaf(av[reg], a.c2, off));
          l_run[j] = fmaf(l_run[j], __builtin_amdgcn_exp2f(fmaf(m_run[j], a.c2, off)), tree_sum16(ev));
          m_run[j] = mn;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NRT; ++j) {
      const float mo = xor32(m_run[j], half), lo = xor32(l_run[j], half);
      const float m = fmaxf(m_run[j], mo);
      float l = 0.f;
      if (m != -INFINITY)
        l = l_run[j] * __builtin_amdgcn_exp2f((m_run[j] - m) * a.c2) + lo * __builtin_amdgcn_exp2f((mo - m) * a.c2);
      if (half == 0) part[wave * NR + j * 32 + l32] = make_float2(m == -INFINITY ? -INFINITY : m * a.c2, l);
    }
    __syncthreads();
    // the workgroup's partial of each row (waves in order)
    for (int r = t; r < a.Rpad; r += NT) {
      float mx = -INFINITY, sx = 0.f;
      for (int w = 0; w < kKrWaves; ++w) mx = fmaxf(mx, part[w * NR + r].x);
      if (mx != -INFINITY)
        for (int w = 0; w < kKrWaves; ++w) {
          const float2 pw = part[w * NR + r];
          if (pw.x != -INFINITY) sx += pw.y * __builtin_amdgcn_exp2f(pw.x - mx);
        }
      a.partials[((int64_t)h * st.total_chunks + gchunk) * a.Rpad + r] = make_float2(mx, sx);
    }
  } else {
    // ---- pass 2: B and Q of the wave's keys, summed over the rows in-lane.
    // The accumulators start at -lse / c2 of their rows, so exp2(c2 * acc) is
    // the softmax probability.
    constexpr int RG = NRT < 2 ? NRT : 2;                  // row tiles per MFMA group
    // accumulator registers of the last query of each group, per row tile
    uint32_t lastm[NRT];
#pragma unroll
    for (int j = 0; j < NRT; ++j) {
      lastm[j] = 0;
      if constexpr (!W32) {
#pragma unroll
        for (int reg = 0; reg < 16; ++reg) {
          const int r = j * 32 + acc_row(reg, half);
          if (r < a.R && (r % W) == W - 1) lastm[j] |= 1u << reg;
        }
      }
    }
    const float inv_gw = 1.f / (float)(a.G * W), inv_g = 1.f / (float)a.G;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 < KT) load_tile(kt + 1);
      const int kbase = k0 + (wave * KT + kt) * 32, key = kbase + l32;
      const bool edge = (kbase + 31 >= k1) || (kbase + 31 > wfirst);
      float bsum = 0.f, qsum = 0.f;
      // the starting values are read again for every group (opaque offset):
      // held across the tiles they would take 16 * NRT registers
      auto seed = [&](int j0, f32x16 *acc) {
        const float *nb = nlc + opaque(4 * half);
#pragma unroll
        for (int j = 0; j < RG; ++j) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float4 v = *reinterpret_cast<const float4 *>(nb + (j0 + j) * 32 + 8 * i);
            acc[j][4 * i + 0] = v.x;
            acc[j][4 * i + 1] = v.y;
            acc[j][4 * i + 2] = v.z;
            acc[j][4 * i + 3] = v.w;
          }
        }
      };
      // acc[j][reg]: row (j0+j)*32 + acc_row(reg, half), key kbase + l32
      auto post = [&](int j0, const f32x16 *acc) {
#pragma unroll
        for (int j = 0; j < RG; ++j) {
          float p[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) p[reg] = __builtin_amdgcn_exp2f(acc[j][reg] * a.c2);
          if (edge) {
#pragma unroll
            for (int reg = 0; reg < 16; ++reg) {
              const int r = (j0 + j) * 32 + acc_row(reg, half);
              const int wr = r < a.R ? r % W : W;
              if (!(key < k1 && key - wfirst <= wr)) p[reg] = 0.f;
            }
          }
          bsum += tree_sum16(p);
          if constexpr (W32) {
            qsum += half ? p[15] : 0.f;
          } else {
#pragma unroll
            for (int reg = 0; reg < 16; ++reg) qsum += ((lastm[j0 + j] >> reg) & 1u) ? p[reg] : 0.f;
          }
        }
      };
      if constexpr (NRT == 2 * RG && W32) {
        // both groups' MFMAs issued before the first group's exps and sums,
        // which then run while the matrix unit works on the second group
        f32x16 acc0[RG], acc1[RG];
        seed(0, acc0);
        tiles(kt, 0, acc0, false);
        seed(RG, acc1);
        tiles(kt, RG, acc1, false);
        post(0, acc0);
        post(RG, acc1);
      } else {
#pragma unroll
        for (int j0 = 0; j0 < NRT; j0 += RG) {
          f32x16 acc[RG];
          seed(j0, acc);
          tiles(kt, j0, acc, false);
          post(j0, acc);
        }
      }
      // E to the history and B out; half h of a wave writes the key tiles of
      // parity h
      bsum += xor32(bsum, half);
      qsum += xor32(qsum, half);
      const int kl = (wave * KT + kt) * 32 + l32;
      if ((kt & 1) == half && key < k1) {
        const float Bv = bsum * inv_gw, Qv = qsum * inv_g;
        const int64_t pos = vrow + key;
        // E (Eq. boundary_residual) to this layer's history slot; the
        // calibration kernel forms L, T and V from the history
        a.ring[a.ring_write * a.ring_stride + pos] = (Qv > Bv) ? (Qv - Bv) : 0.f;
        a.vec_B[pos] = Bv;
        cb[kl] = Bv;
      }
    }
    __syncthreads();

    // B histogram of the chunk's candidates, as in the streaming pass
    unsigned *hist = reinterpret_cast<unsigned *>(qbuf);
    const int ncnd = max(0, min(k1, wfirst) - k0);
    int blo = kHBins, bhi = -1;
    for (int p = t; p < ncnd; p += NT) {
      const int q = hbin(float_key(cb[p]));
      blo = min(blo, q);
      bhi = max(bhi, q);
    }
    blo = __reduce_min_sync(~0ull, blo);
    bhi = __reduce_max_sync(~0ull, bhi);
    int *mm = reinterpret_cast<int *>(part);
    if (lane == 0) { mm[wave] = blo; mm[kKrWaves + wave] = bhi; }
    __syncthreads();
    blo = kHBins;
    bhi = -1;
    for (int w = 0; w < kKrWaves; ++w) {
      blo = min(blo, mm[w]);
      bhi = max(bhi, mm[kKrWaves + w]);
    }
    for (int q = blo + t; q <= bhi; q += NT) hist[q] = 0u;
    __syncthreads();
    for (int p = t; p < ncnd; p += NT) atomicAdd(&hist[hbin(float_key(cb[p]))], 1u);
    __syncthreads();
    const int copy = (h * st.total_chunks + gchunk) % kHCopies;
    unsigned *gh = a.hist_B + (((int64_t)b * a.Hkv + h) * kHCopies + copy) * kHBins;
    for (int q = blo + t; q <= bhi; q += NT) {
      const unsigned cnt = hist[q];
      if (cnt) atomicAdd(&gh[q], cnt);
    }
  }
}

// two workgroups per CU: at most 256 registers per wave
template <int MODE, int D, bool W32, int NRT>
__global__ __launch_bounds__(64 * kKrWaves, 2) void k_krpass(PassArgs a, SeqTable st) {
  krpass_body<MODE, D, W32, NRT>(a, st, blockIdx.x, blockIdx.y);
}

// Pass 2 of one layer (a2) and pass 1 of the next (a1) in one grid: the first
// total_chunks columns of workgroups take a2, the others a1.  Both layers
// share the batch (one SeqTable); the two halves touch disjoint buffers
// (pass 2 reads the merged normalisers and writes E, B and the B histogram;
// pass 1 writes the per-chunk partials).  One launch instead of two, and the
// workgroups of pass 1 fill the CUs that pass 2 leaves idle at its end.
template <int D, bool W32, int NRT>
__global__ __launch_bounds__(64 * kKrWaves, 2) void k_krdual(PassArgs a2, PassArgs a1, SeqTable st) {
  if ((int)blockIdx.x < st.total_chunks)
    krpass_body<PASS_FUSED, D, W32, NRT>(a2, st, blockIdx.x, blockIdx.y);
  else
    krpass_body<PASS_LSE, D, false, NRT>(a1, st, blockIdx.x - st.total_chunks, blockIdx.y);
}

template <int D, bool W32, int NRT>
static hipError_t launch_dual_t(const PassArgs &a2, const PassArgs &a1, const SeqTable &st,
                                hipStream_t s) {
  const int lds = kr_lds_bytes(true, D, a2.Rpad);
  if (lds > kLdsBytes) return hipErrorInvalidValue;
  auto kern = k_krdual<D, W32, NRT>;
  allow_lds(kern, lds);
  hipLaunchKernelGGL(kern, dim3(2 * st.total_chunks, a2.Hkv), dim3(64 * kKrWaves), lds, s, a2, a1,
                     st);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_dual_d(bool w32, const PassArgs &a2, const PassArgs &a1, const SeqTable &st,
                                hipStream_t s) {
  if (kr_row_tiles(a2.Rpad) == 2)
    return w32 ? launch_dual_t<D, true, 2>(a2, a1, st, s) : launch_dual_t<D, false, 2>(a2, a1, st, s);
  return w32 ? launch_dual_t<D, true, 4>(a2, a1, st, s) : launch_dual_t<D, false, 4>(a2, a1, st, s);
}

template <int MODE, int D, bool W32, int NRT>
static hipError_t launch_kr_t(const PassArgs &a, const SeqTable &st, hipStream_t s) {
  const int lds = kr_lds_bytes(true, D, a.Rpad);
  if (lds > kLdsBytes) return hipErrorInvalidValue;
  auto kern = k_krpass<MODE, D, W32, NRT>;
  allow_lds(kern, lds);
  hipLaunchKernelGGL(kern, dim3(st.total_chunks, a.Hkv), dim3(64 * kKrWaves), lds, s, a, st);
  return hipGetLastError();
}

template <int MODE, int D>
static hipError_t launch_kr_d(bool w32, const PassArgs &a, const SeqTable &st, hipStream_t s) {
  if (kr_row_tiles(a.Rpad) == 2)
    return w32 ? launch_kr_t<MODE, D, true, 2>(a, st, s) : launch_kr_t<MODE, D, false, 2>(a, st, s);
  return w32 ? launch_kr_t<MODE, D, true, 4>(a, st, s) : launch_kr_t<MODE, D, false, 4>(a, st, s);
}

bool kr_supported(bool bf16, int head_dim, int rpad) {
  return bf16 && kr_row_tiles(rpad) > 0 && kr_lds_bytes(bf16, head_dim, rpad) <= kLdsBytes;
}

hipError_t launch_krdual(bool bf16, int head_dim, bool w32, const PassArgs &a2, const PassArgs &a1,
                         const SeqTable &st, hipStream_t s) {
  if (!kr_supported(bf16, head_dim, a2.Rpad) || a1.Rpad != a2.Rpad) return hipErrorInvalidValue;
  return head_dim == 128 ? launch_dual_d<128>(w32, a2, a1, st, s) : launch_dual_d<64>(w32, a2, a1, st, s);
}

hipError_t launch_krpass(int mode, bool bf16, int head_dim, bool w32, const PassArgs &a,
                         const SeqTable &st, hipStream_t s) {
  if (!kr_supported(bf16, head_dim, a.Rpad) || (mode != PASS_LSE && mode != PASS_FUSED))
    return hipErrorInvalidValue;
  if (mode == PASS_LSE)
    return head_dim == 128 ? launch_kr_d<PASS_LSE, 128>(false, a, st, s) : launch_kr_d<PASS_LSE, 64>(false, a, st, s);
  return head_dim == 128 ? launch_kr_d<PASS_FUSED, 128>(w32, a, st, s) : launch_kr_d<PASS_FUSED, 64>(w32, a, st, s);
}

// ---------------------------------------------------------------- single-read pass
// One read of K per layer (bf16 keys, up to 128 window rows).  A workgroup of
// kKrWaves waves holds kr_keys() keys of one KV head, loaded straight into
// registers in the MFMA operand layout, as in the key-register passes.
//
//  * Pass 1 (D = K Q^T, a lane per query row) forms the probabilities of each
//    key tile against the row's running max, which both halves of the wave
//    share, and keeps them in registers as fp16 (the key registers of a tile
//    are free once its MFMAs have run, so the register count of keys plus
//    probabilities stays that of the keys).  What is stored is p - p_min
//    times 2^15, p_min the smallest probability of the row in the tile: never
//    less precise than p itself (0 <= p - p_min <= p), and far more precise
//    where attention is near uniform and the residual Q - B cancels.  The max
//    each tile used and p_min go to LDS.
//  * The chunks of a (sequence, KV head) meet once: each publishes its
//    per-row (max, sum) partial through to memory (agent-scope stores),
//    counts itself on the group's arrival counter; the last to arrive merges
//    all partials in chunk order into the row normalisers and publishes them,
//    and the others poll for them.  The last workgroup to finish reading
//    resets the counters and the published words at its end.
//    The waits are bounded: one that runs out sets the error word and goes
//    on.  Workgroups are dispatched in grid order, chunk-major with the KV
//    heads innermost, so the groups not yet complete are those of one
//    sequence; the host launches this pass only when their chunks fit on the
//    GPU at once.
//  * Pass 2 turns each stored 32x32 block around with two MFMAs against the
//    identity (a lane per key, the rows in registers) and sums its rows,
//    each weighted by exp2(tile max - lse) / 2^15, with two more MFMAs whose
//    other operand holds the row weights in fp16 as high and low parts; it
//    adds the tile's sum of the weighted p_min: B and Q without a second
//    read of K or a second exp.  The tail (E to the history, B out, the B
//    histogram) is that of the key-register pass 2.
constexpr float kPScaleLog2 = 15.f;          // stored probabilities are p * 2^15 (<= 2^15)
constexpr int kWScaleLog2 = 12;              // pass 2's fp16 row factors are scaled by 2^(15 + this)
// The factor operand's columns lie a multiple of 4 KiB plus 32 bytes apart,
// so that the four lanes that read the same rows of different columns use
// different LDS banks.
constexpr int kWPad = 16;
constexpr unsigned kMeetSpin = 1u << 20;     // polls of a published word before giving up

__device__ __forceinline__ void store_agent(float2 *p, float2 v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long *>(p), __builtin_bit_cast(unsigned long long, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_agent(const float2 *p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const unsigned long long *>(p),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
__device__ __forceinline__ void store_agent(float *p, float v) {
  __hip_atomic_store(reinterpret_cast<unsigned *>(p), __builtin_bit_cast(unsigned, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_agent(const float *p) {
  return __builtin_bit_cast(float, __hip_atomic_load(reinterpret_cast<const unsigned *>(p), __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT));
}

// A device-scope atomic add whose old value is awaited only by await_vm():
// the compiler's own form of a one-lane atomic waits for the return at once.
// The vector atomic is the form the compiler emits for a relaxed agent-scope
// add (old value returned); the compiler does not count it among its own
// outstanding loads, which only makes its later waits stricter.
__device__ __forceinline__ unsigned atomic_add_deferred(unsigned *p, unsigned v) {
  unsigned r;
  asm volatile("global_atomic_add %0, %1, %2, off sc0" : "=v"(r) : "v"(p), "v"(v) : "memory");
  return r;
}
__device__ __forceinline__ void await_vm(unsigned &r) {
  asm volatile("s_waitcnt vmcnt(0)" : "+v"(r) : : "memory");
}

__device__ __forceinline__ void pin8(unsigned (&v)[8]) {
  asm volatile("" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
               "+v"(v[7]));
}

__device__ __forceinline__ unsigned pack_f16(float lo, float hi) {
  typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
  const f16x2 v = {(_Float16)lo, (_Float16)hi};
  return __builtin_bit_cast(unsigned, v);
}

// LDS map of a single-read workgroup (bytes), NR = 32 * row tiles:
//   qbuf  max(NR * ROWB, 4 * kHBins)      window queries; the B histogram after pass 1
//   part  max(kKrWaves * NR, NT) float2   per-wave row partials; merge scratch
//   fac   kKrWaves * KT * NR floats       the max each tile used
//   rmn   kKrWaves * KT * NR floats       p_min * 2^15 of each row in each tile
//   lse   NR floats                       merged row normalisers (log2 units)
//   wf    4 * (kKrWaves * KT * NR + kWPad)  the row factors as pass 2's operand
//         + 32 fp16                       (four columns: high and low parts, and
//                                         the same on the last-query rows only;
//                                         then zeros)
int single_lds_bytes(int head_dim, int rpad) {
  const int nr = 32 * kr_row_tiles(rpad), rowb = head_dim * 2, kpw = kr_keys(true, head_dim);
  const int kt = kpw / (32 * kKrWaves);
  return std::max(nr * rowb, 4 * kHBins) + 8 * std::max(kKrWaves * nr, 64 * kKrWaves) +
         8 * kKrWaves * kt * nr + 4 * nr + 2 * (4 * (kKrWaves * kt * nr + kWPad) + 32);
}

template <int D, bool W32, int NRT>
__global__ __launch_bounds__(64 * kKrWaves, 2) void k_single(PassArgs a, SeqTable st) {
  using C = PassCfg<true, D>;
  constexpr int NU = C::NU, KT = KrCfg<true, D>::KT, KPW = KrCfg<true, D>::KPW;
  constexpr int NT = 64 * kKrWaves, NR = 32 * NRT;
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_go;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63, half = lane >> 5, l32 = lane & 31;
  const int h = (int)blockIdx.x % a.Hkv, gchunk = (int)blockIdx.x / a.Hkv;
  const int b = find_seq(st, gchunk);
  const int c = gchunk - st.chunk_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int nch = st.chunk_base[b + 1] - st.chunk_base[b];
  const int k0 = c * KPW, k1 = min(n, k0 + KPW);
  const int W = a.W, wfirst = n - W;
  const int64_t vrow = (int64_t)h * a.T + st.cu[b];      // [Hkv, T] index of the sequence's position 0
  const int grp = b * a.Hkv + h;

  unsigned char *qbuf = smem;
  float2 *part = reinterpret_cast<float2 *>(smem + max(NR * C::ROWB, 4 * kHBins));
  float *fac = reinterpret_cast<float *>(part + max(kKrWaves * NR, NT));
  float *rmn = fac + kKrWaves * KT * NR;
  float *lse = rmn + kKrWaves * KT * NR;
  _Float16 *wf = reinterpret_cast<_Float16 *>(lse + NR);   // [4][kKrWaves * KT * NR] then 32 zeros

  // ---- loads: the window queries, the first key tile, and once the queries
  // are in LDS the other key tiles (as in the key-register passes)
  constexpr int QP = NR * C::PIECES / NT;
  u32x4 qv[QP];
#pragma unroll
  for (int j = 0; j < QP; ++j) {
    const int i = t + j * NT, row = i / C::PIECES, pc = i % C::PIECES;
    const int rr = min(row, a.R - 1), g = rr / W, w = rr - g * W;
    qv[j] = *reinterpret_cast<const u32x4 *>(static_cast<const unsigned char *>(a.q) +
        ((int64_t)(b * W + w) * a.Hq + (int64_t)h * a.G + g) * C::ROWB + 16 * pc);
  }
  const int64_t kstride = (int64_t)a.Hkv * C::ROWB;
  const unsigned char *kb = static_cast<const unsigned char *>(a.k) +
                            ((int64_t)st.cu[b] * a.Hkv + h) * C::ROWB + 16 * half;
  u32x4 kr[KT][NU];
  auto load_tile = [&](int kt) {
    const int key = min(k0 + (wave * KT + kt) * 32 + l32, k1 - 1);
    const unsigned char *kp = kb + (int64_t)key * kstride;
#pragma unroll
    for (int u = 0; u < NU; ++u) kr[kt][u] = *reinterpret_cast<const u32x4 *>(kp + 32 * u);
  };
  asm volatile("" ::: "memory");
  load_tile(0);
  asm volatile("" ::: "memory");
#pragma unroll
  for (int j = 0; j < QP; ++j) pin(qv[j]);
#pragma unroll
  for (int j = 0; j < QP; ++j) {
    const int i = t + j * NT, row = i / C::PIECES, pc = i % C::PIECES;
    *reinterpret_cast<u32x4 *>(qbuf + row * C::ROWB + 16 * (pc ^ (row & C::SWM))) = qv[j];
  }
  // the zeros that pass 2's idle factor lanes read
  if (t < 32) wf[4 * (kKrWaves * KT * NR + kWPad) + t] = (_Float16)0.f;
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  // each later tile's keys are requested when the wave starts that tile
  // (the other waves of the SIMD cover the wait).  Requested further ahead,
  // every workgroup's requests go out at once and the second workgroup of
  // each CU receives its keys last: about 1.5 us later in the launch with
  // two tiles ahead, 0.5 us with one

  int koff[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) koff[u] = l32 * C::ROWB + 16 * ((2 * u + half) ^ (l32 & C::SWM));

  // ---- pass 1: probabilities of each tile against the running row max, two
  // row tiles at a time (their accumulators and query fragments are what the
  // stored probabilities leave of the register file); the max each tile used
  // goes to LDS
  constexpr int RG = NRT < 2 ? NRT : 2;
  unsigned pk[KT][NRT][8];          // fp16 pairs: keys acc_row(2q, half), acc_row(2q + 1, half)
  float m_run[NRT], l_run[NRT];
#pragma unroll
  for (int j = 0; j < NRT; ++j) { m_run[j] = -INFINITY; l_run[j] = 0.f; }
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    if (kt > 0) load_tile(kt);
    const int kbase = k0 + (wave * KT + kt) * 32;
    const bool edge = (kbase + 31 >= k1) || (kbase + 31 > wfirst);
#pragma unroll
    for (int j0 = 0; j0 < NRT; j0 += RG) {
      f32x16 acc[RG];
#pragma unroll
      for (int j = 0; j < RG; ++j) acc[j] = f32x16{};
      {
        u32x4 qf[2][RG];
#pragma unroll
        for (int j = 0; j < RG; ++j)
          qf[0][j] = *reinterpret_cast<const u32x4 *>(qbuf + (j0 + j) * 32 * C::ROWB + koff[0]);
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          if (u + 1 < NU) {
#pragma unroll
            for (int j = 0; j < RG; ++j)
              qf[(u + 1) & 1][j] = *reinterpret_cast<const u32x4 *>(qbuf + (j0 + j) * 32 * C::ROWB + koff[u + 1]);
          }
#pragma unroll
          for (int j = 0; j < RG; ++j) acc[j] = mfma_unit<true>(kr[kt][u], qf[u & 1][j], acc[j]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // acc[j][reg]: key kbase + acc_row(reg, half), row (j0 + j)*32 + l32.
      // Tiles away from the sequence end and the window take the unmasked
      // form; the two forms are separate branches, which also keeps the
      // compiler from issuing every tile's MFMAs ahead of the exps.
      auto post = [&](bool masked) {
#pragma unroll
        for (int jj = 0; jj < RG; ++jj) {
          const int j = j0 + jj;
          const int r = j * 32 + l32;
          float av[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) av[reg] = acc[jj][reg];
          if (masked) {
            const int tpos = wfirst + (r < a.R ? r % W : W - 1);
#pragma unroll
            for (int reg = 0; reg < 16; ++reg) {
              const int key = kbase + acc_row(reg, half);
              if (!(key < k1 && key <= tpos)) av[reg] = -INFINITY;
            }
          }
          float mt = tree_max16(av), lo = tree_min16(av);
          mt = fmaxf(mt, xor32(mt, half));
          lo = fminf(lo, xor32(lo, half));
          const float mn = fmaxf(m_run[j], mt);
          const float off = (mn == -INFINITY ? 0.f : -mn * a.c2) + kPScaleLog2;
          float ev[16];
#pragma unroll
          for (int reg = 0; reg < 16; ++reg) ev[reg] = __builtin_amdgcn_exp2f(fmaf(av[reg], a.c2, off));
          l_run[j] = fmaf(l_run[j], __builtin_amdgcn_exp2f(fmaf(m_run[j], a.c2, off - kPScaleLog2)),
                          tree_sum16(ev) * (1.f / 32768.f));
          m_run[j] = mn;
          // the tile's smallest probability of the row (0 when a key of the
          // tile is masked), the same exp as its element's
          const float pmin = __builtin_amdgcn_exp2f(fmaf(lo, a.c2, off));
          if (half == 0) {
            fac[(wave * KT + kt) * NR + r] = mn;
            rmn[(wave * KT + kt) * NR + r] = pmin;
          }
#pragma unroll
          for (int q = 0; q < 8; ++q) pk[kt][j][q] = pack_f16(ev[2 * q] - pmin, ev[2 * q + 1] - pmin);
          // the packed probabilities as formed here: keeps the compiler
          // from sinking the exps to their uses in pass 2
          pin8(pk[kt][j]);
        }
      };
      if (edge) post(true); else post(false);
    }
  }
  // the wave's (max, sum) per row (log2 units; both halves share the max)
#pragma unroll
  for (int j = 0; j < NRT; ++j) {
    const float l = l_run[j] + xor32(l_run[j], half);
    if (half == 0)
      part[wave * NR + j * 32 + l32] = make_float2(m_run[j] == -INFINITY ? -INFINITY : m_run[j] * a.c2, l);
  }
  __syncthreads();
  // every wave is past pass 1: the window queries' space holds the B
  // histogram of the chunk from here (cleared now, counted in pass 2's tail;
  // the barriers of the meeting order the two)
  unsigned *hist = reinterpret_cast<unsigned *>(qbuf);
  for (int q = 4 * t; q < kHBins; q += 4 * NT) *reinterpret_cast<uint4 *>(hist + q) = make_uint4(0u, 0u, 0u, 0u);
  // the workgroup's partial of each row (waves in order), written through
  const int64_t pbase = ((int64_t)h * st.total_chunks + st.chunk_base[b]) * a.Rpad;
  if (t < a.Rpad) {
    float mx = -INFINITY, sx = 0.f;
    for (int w = 0; w < kKrWaves; ++w) mx = fmaxf(mx, part[w * NR + t].x);
    if (mx != -INFINITY)
      for (int w = 0; w < kKrWaves; ++w) {
        const float2 pw = part[w * NR + t];
        if (pw.x != -INFINITY) sx += pw.y * __builtin_amdgcn_exp2f(pw.x - mx);
      }
    store_agent(a.partials + pbase + (int64_t)c * a.Rpad + t, make_float2(mx, sx));
  }
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  __syncthreads();

  // ---- the meeting of the chunks of (b, h).  The last workgroup to arrive
  // merges the group's partials in chunk order and publishes the row
  // normalisers; the others poll their rows of the published words (the
  // complement of the float's bits, never 0 for a finite value or +inf, so
  // 0 means not yet), backing off between polls.
  unsigned *arrive = a.sync + kSyncStride * grp, *done = arrive + 1;
  unsigned *pub = a.bcast + (int64_t)grp * a.Rpad;
  if (t == 0) {
    const unsigned prev = __hip_atomic_fetch_add(arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_go = prev + 1 == (unsigned)nch;
  }
  __syncthreads();
  if (s_go) {
    // thread t takes row t % Rpad over the chunks congruent to t / Rpad,
    // 32 loads in flight (every chunk of a 32K sequence at Rpad = 128)
    constexpr int FL = 32;
    const int parts = NT / a.Rpad, row = t % a.Rpad, pp = t / a.Rpad;
    float mm = -INFINITY, ll = 0.f;
    if (pp < parts) {
      const float2 *src = a.partials + pbase + row;
      for (int c0 = pp; c0 < nch; c0 += FL * parts) {
        float2 v[FL];
#pragma unroll
        for (int j = 0; j < FL; ++j) v[j] = load_agent(src + (int64_t)min(c0 + j * parts, nch - 1) * a.Rpad);
#pragma unroll
        for (int j = 0; j < FL; ++j)
          if (c0 + j * parts >= nch) v[j] = make_float2(-INFINITY, 0.f);
        float mb = mm;
#pragma unroll
        for (int j = 0; j < FL; ++j) mb = fmaxf(mb, v[j].x);
        if (mb != -INFINITY) {
          float acc = (mm == -INFINITY) ? 0.f : ll * __builtin_amdgcn_exp2f(mm - mb);
#pragma unroll
          for (int j = 0; j < FL; ++j)
            if (v[j].x != -INFINITY) acc += v[j].y * __builtin_amdgcn_exp2f(v[j].x - mb);
          ll = acc;
          mm = mb;
        }
      }
    }
    part[t] = make_float2(mm, ll);
    __syncthreads();
    if (t < a.Rpad) {
      float mx = -INFINITY, sx = 0.f;
      for (int q = 0; q < parts; ++q) mx = fmaxf(mx, part[q * a.Rpad + t].x);
      if (mx != -INFINITY)
        for (int q = 0; q < parts; ++q) {
          const float2 pq = part[q * a.Rpad + t];
          if (pq.x != -INFINITY) sx += pq.y * __builtin_amdgcn_exp2f(pq.x - mx);
        }
      const float l2 = (t < a.R) ? mx + log2f(sx) : INFINITY;
      lse[t] = l2;
      __hip_atomic_store(pub + t, ~__builtin_bit_cast(unsigned, l2), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      a.lse2[(int64_t)grp * a.Rpad + t] = l2;
      if (a.lse_user && t < a.R) {
        const int g = t / W, w = t - g * W;
        a.lse_user[((int64_t)b * a.Hq + (int64_t)h * a.G + g) * W + w] = l2 * kLn2;
      }
    }
  } else if (t < a.Rpad) {
    unsigned v, polls = 0;
    while ((v = __hip_atomic_load(pub + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == 0u) {
      __builtin_amdgcn_s_sleep(16);
      if (++polls == kMeetSpin) {
        __hip_atomic_store(a.sync + kSyncStride * a.sync_groups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
    lse[t] = __builtin_bit_cast(float, ~v);
  }
  if (t >= a.Rpad && t < NR) lse[t] = INFINITY;   // rows of the last tile past Rpad: factor 0
  __syncthreads();
  // the normalisers are read: count this workgroup out of the meeting now;
  // the last of the group to get here clears the counters and the published
  // words for the next launch, at its end (the count's return is awaited
  // there)
  unsigned done_prev = 0;
  if (t == 0) done_prev = atomic_add_deferred(done, 1u);

  // ---- row factors of the wave's own tiles (each wave reads and writes only
  // its tiles' rows, so no workgroup barrier): exp2(tile max - lse) / 2^15,
  // zero for pad rows (lse = +inf) and rows with no key so far (max = -inf;
  // exp2 of -inf is 0).  The same times 2^(15 + kWScaleLog2) in fp16 as a
  // high and a low part (their sum within about 2^-22 of it) form pass 2's
  // contraction operand for B; Q takes the last-query rows: with a 32-query
  // window, row 31 of every row tile, whose factors pass 2 applies in fp32
  // (fq), else two more operand columns on those rows only.  Per tile also
  // the sums over the rows of factor * p_min (into B) and over the
  // last-query rows (into Q), in a fixed order.
  constexpr int NE = kKrWaves * KT * NR;
  constexpr int WS = NE + kWPad;    // column stride of the factor operand
  constexpr int RL = NR / 64;       // rows per lane
  float cB[KT], cQ[KT];
  float fq[KT][NRT];                // W32: the factors of rows 32 j + 31
  {
    float l2r[RL];
    bool lastq[RL];
#pragma unroll
    for (int q = 0; q < RL; ++q) {
      const int r = lane + 64 * q;
      l2r[q] = lse[r];
      lastq[q] = r < a.R && (r % W) == W - 1;
    }
    constexpr float kWScale = (float)(1 << (15 + kWScaleLog2));
    static_assert(KT == 4, "the p_min sums of a wave are eight values");
    float sx[8];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      float sb = 0.f, sq = 0.f;
#pragma unroll
      for (int q = 0; q < RL; ++q) {
        const int e = (wave * KT + kt) * NR + lane + 64 * q;
        const float m = fac[e], pm = rmn[e];
        const float f = __builtin_amdgcn_exp2f(fmaf(m, a.c2, -l2r[q]) - kPScaleLog2);
        const float fs = f * kWScale;
        const _Float16 hi = (_Float16)fs;
        const _Float16 lo = (_Float16)(fs - (float)hi);
        wf[e] = hi;
        wf[WS + e] = lo;
        if constexpr (!W32) {
          wf[2 * WS + e] = lastq[q] ? hi : (_Float16)0.f;
          wf[3 * WS + e] = lastq[q] ? lo : (_Float16)0.f;
        }
        const float v = f * pm;
        sb += v;
        sq += lastq[q] ? v : 0.f;
        if constexpr (W32) {
          // rows 64 q + 31 and 64 q + 63 are row tiles 2q and 2q + 1's row 31
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
            if (2 * q + jj < NRT)
              fq[kt][2 * q + jj] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), 31 + 32 * jj));
        }
      }
      sx[kt] = sb;
      sx[4 + kt] = sq;
    }
    float ss[8];
    wave_sum8(sx, ss, lane);
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      cB[kt] = ss[kt];
      cQ[kt] = ss[4 + kt];
    }
  }

  // ---- pass 2: B and Q of the wave's keys from the stored probabilities,
  // on the matrix cores.  Per block (kt, j): two fp16 MFMAs against identity
  // operands transpose the block (a lane per key; the A operand of block
  // (kt, j) holds, in lane l, the probabilities of row l % 32 for keys
  // 4h + (s & 3) + 8 (s >> 2) of k-slot 8h + s, h = l / 32, and lane l of
  // the identity holds a 1 where its column l % 32 is that key), and two
  // 16x16x32 MFMAs contract it over the rows with the row factors: the
  // factor columns (high part, low part, and without a 32-query window the
  // two on the last-query rows only) in the A operand, the transposed block
  // in the B operand, so that the output registers of lane l < 32 are those
  // sums for key l.
  u32x4 idop[2];
  {
    const int np = l32 & 15, aa = np >> 3, bb = (np >> 2) & 1, cc = np & 3, slot = 4 * aa + cc;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2) {
      unsigned w4[4] = {0u, 0u, 0u, 0u};
      if ((l32 >> 4) == kb2 && bb == half) w4[slot >> 1] = (slot & 1) ? 0x3C000000u : 0x00003C00u;
      idop[kb2] = u32x4{w4[0], w4[1], w4[2], w4[3]};
    }
  }
  typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
  // The factor operand of the 16x16x32 contractions: lane l holds column
  // m = l % 16 for k-slots 8 g + i (g = l / 16), and lane group g of the B
  // operand holds keys 16 (g & 1) + n (n = l % 16) of half g >> 1.  Output
  // rows 0..3 take the factor columns over the lane groups of keys 0..15,
  // rows 4..7 over those of keys 16..31; the other lanes (and, with a
  // 32-query window, columns 2 and 3) read zeros.
  const int g16 = lane >> 4, m16 = lane & 15;
  const bool wact = ((g16 & 1) ? (m16 >= 4 && m16 < 8) : (m16 < 4)) && (!W32 || (m16 & 3) < 2);
  const _Float16 *wcol = wact ? wf + (m16 & 3) * WS : wf + 4 * WS;
  const int wstep = wact ? 1 : 0;
  auto transpose = [&](int kt, int j) {
    f32x16 d = f32x16{};
    d = __builtin_amdgcn_mfma_f32_32x32x16_f16(
        __builtin_bit_cast(f16x8, u32x4{pk[kt][j][0], pk[kt][j][1], pk[kt][j][2], pk[kt][j][3]}),
        __builtin_bit_cast(f16x8, idop[0]), d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_32x32x16_f16(
        __builtin_bit_cast(f16x8, u32x4{pk[kt][j][4], pk[kt][j][5], pk[kt][j][6], pk[kt][j][7]}),
        __builtin_bit_cast(f16x8, idop[1]), d, 0, 0, 0);
    return d;
  };
  // blocks in order kt-major; each block's transposes are issued before the
  // previous block's contraction, which waits on their results otherwise
  f32x4 acc2[KT];
  float qacc[KT];                   // W32: Q of key l % 32 in the lanes of the second half
  constexpr int NB = KT * NRT;
  f32x16 dn = transpose(0, 0);
#pragma unroll
  for (int blk = 0; blk < NB; ++blk) {
    const int kt = blk / NRT, j = blk % NRT;
    const f32x16 d = dn;
    if (blk + 1 < NB) dn = transpose((blk + 1) / NRT, (blk + 1) % NRT);
    // register 15 of the second half's lanes is row acc_row(15, 1) = 31
    if constexpr (W32) qacc[kt] = fmaf(fq[kt][j], d[15], j == 0 ? 0.f : qacc[kt]);
    // d[reg]: row j*32 + acc_row(reg, half), key kbase + l32: k-slot 8h + i
    // of the two contractions is row acc_row(i, h) and acc_row(8 + i, h)
    f16x8 bo[2];
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) bo[g][i] = (_Float16)d[8 * g + i];
    // the factor operand: rows acc_row(0..7, h) are two runs of four,
    // 4h + 0..3 and 8 + 4h + 0..3 (and 16, 24 further for the second)
    const _Float16 *wr = wcol + wstep * ((wave * KT + kt) * NR + j * 32 + 4 * (g16 >> 1));
    f16x8 ao[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const uint2 lo4 = *reinterpret_cast<const uint2 *>(wr + wstep * (16 * g));
      const uint2 hi4 = *reinterpret_cast<const uint2 *>(wr + wstep * (16 * g + 8));
      ao[g] = __builtin_bit_cast(f16x8, u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
    }
    if (j == 0) acc2[kt] = f32x4{};
    acc2[kt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ao[0], bo[0], acc2[kt], 0, 0, 0);
    acc2[kt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ao[1], bo[1], acc2[kt], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  const float inv_gw = 1.f / (float)(a.G * W), inv_g = 1.f / (float)a.G;
  constexpr float kUnscale = 1.f / (float)(1 << (15 + kWScaleLog2));
  // B, E, and the B histogram of the chunk's candidates (keys before the
  // window) with the range of bins it touched
  int blo = kHBins, bhi = -1;
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    const int key = k0 + (wave * KT + kt) * 32 + l32;
    float qw = 0.f;
    if constexpr (W32) qw = xor32(qacc[kt], half);
    if (half == 0 && key < k1) {
      const float bs = fmaf(acc2[kt][0] + acc2[kt][1], kUnscale, cB[kt]);
      const float qs = W32 ? qw + cQ[kt] : fmaf(acc2[kt][2] + acc2[kt][3], kUnscale, cQ[kt]);
      const float Bv = bs * inv_gw, Qv = qs * inv_g;
      const int64_t pos = vrow + key;
      // E (Eq. boundary_residual) to this layer's history slot
      a.ring[a.ring_write * a.ring_stride + pos] = (Qv > Bv) ? (Qv - Bv) : 0.f;
      a.vec_B[pos] = Bv;
      if (key < wfirst) {
        const int q = hbin(float_key(Bv));
        atomicAdd(&hist[q], 1u);
        blo = min(blo, q);
        bhi = max(bhi, q);
      }
    }
  }
  blo = __reduce_min_sync(~0ull, blo);
  bhi = __reduce_max_sync(~0ull, bhi);
  int *mm2 = reinterpret_cast<int *>(part);
  if (lane == 0) { mm2[wave] = blo; mm2[kKrWaves + wave] = bhi; }
  if (t == 0) {
    await_vm(done_prev);
    s_go = done_prev + 1 == (unsigned)nch;
    if (s_go) {
      __hip_atomic_store(arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  if (s_go && t < a.Rpad) __hip_atomic_store(pub + t, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  blo = kHBins;
  bhi = -1;
  for (int w = 0; w < kKrWaves; ++w) {
    blo = min(blo, mm2[w]);
    bhi = max(bhi, mm2[kKrWaves + w]);
  }
  const int copy = (h * st.total_chunks + gchunk) % kHCopies;
  unsigned *gh = a.hist_B + (((int64_t)b * a.Hkv + h) * kHCopies + copy) * kHBins;
  for (int q = blo + t; q <= bhi; q += NT) {
    const unsigned cnt = hist[q];
    if (cnt) atomicAdd(&gh[q], cnt);
  }
}

template <int D, bool W32, int NRT>
static hipError_t launch_single_t(const PassArgs &a, const SeqTable &st, hipStream_t s) {
  const int lds = single_lds_bytes(D, a.Rpad);
  if (lds > kLdsBytes / 2) return hipErrorInvalidValue;
  auto kern = k_single<D, W32, NRT>;
  allow_lds(kern, lds);
  hipLaunchKernelGGL(kern, dim3(st.total_chunks * a.Hkv), dim3(64 * kKrWaves), lds, s, a, st);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_single_d(bool w32, const PassArgs &a, const SeqTable &st, hipStream_t s) {
  if (kr_row_tiles(a.Rpad) == 2)
    return w32 ? launch_single_t<D, true, 2>(a, st, s) : launch_single_t<D, false, 2>(a, st, s);
  return w32 ? launch_single_t<D, true, 4>(a, st, s) : launch_single_t<D, false, 4>(a, st, s);
}

hipError_t launch_single(int head_dim, bool w32, const PassArgs &a, const SeqTable &st, hipStream_t s) {
  if (!kr_supported(true, head_dim, a.Rpad) || !a.sync || !a.bcast) return hipErrorInvalidValue;
  return head_dim == 128 ? launch_single_d<128>(w32, a, st, s) : launch_single_d<64>(w32, a, st, s);
}

int single_resident_blocks(int head_dim, int rpad) {
  const int lds = single_lds_bytes(head_dim, rpad);
  int per_cu = 0;
  hipError_t e;
  if (head_dim == 128)
    e = kr_row_tiles(rpad) == 2
            ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_single<128, true, 2>, 64 * kKrWaves, lds)
            : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_single<128, true, 4>, 64 * kKrWaves, lds);
  else
    e = kr_row_tiles(rpad) == 2
            ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_single<64, true, 2>, 64 * kKrWaves, lds)
            : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_single<64, true, 4>, 64 * kKrWaves, lds);
  if (e != hipSuccess) return 0;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  return per_cu * cus;
}

// ---------------------------------------------------------------- block helpers
// Workgroup barrier for LDS traffic: waits for this wave's LDS operations
// only.  The fence of __syncthreads also waits for every global load and
// store the wave has in flight, which the select kernels never need: none
// of them reads global memory another of its threads wrote in the same
// launch; their threads exchange data through LDS only.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
// Shared scratch of the block-wide primitives for NT threads.
template <int NT>
struct SelSharedT {
  unsigned hist[kHistBins];
  unsigned red_u[NT / 64], red_u2[NT / 64];
  double red_d[4][NT / 64];
  unsigned bc_u[4];
  double bc_d[4];
  int bc_i[4];
};

// Xor lane exchange inside each 32-lane half through ds_swizzle (immediate
// pattern, no index registers).
template <int X>
__device__ __forceinline__ unsigned swz(unsigned v) {
  return (unsigned)__builtin_amdgcn_ds_swizzle((int)v, (X << 10) | 0x1f);
}

// Wave-wide scans and reductions through DPP lane moves (GFX9 encodings):
// row_shr:n (0x110 + n) shifts lanes by n inside each 16-lane row,
// row_bcast:15 (0x142) copies lane 15 of a row into the next row and
// row_bcast:31 (0x143) lane 31 into rows 2 and 3.  Lanes with no source, or
// outside the row mask, receive `id`.  After the six steps lane i holds the
// inclusive scan over lanes 0..i; lane 63 the whole wave.
template <int CTRL, int ROWS>
__device__ __forceinline__ unsigned dpp_u(unsigned id, unsigned v) {
  return (unsigned)__builtin_amdgcn_update_dpp((int)id, (int)v, CTRL, ROWS, 0xf, false);
}
template <typename Op>
__device__ __forceinline__ unsigned wave_scan_u(unsigned v, unsigned id, Op op) {
  v = op(v, dpp_u<0x111, 0xf>(id, v));
  v = op(v, dpp_u<0x112, 0xf>(id, v));
  v = op(v, dpp_u<0x114, 0xf>(id, v));
  v = op(v, dpp_u<0x118, 0xf>(id, v));
  v = op(v, dpp_u<0x142, 0xa>(id, v));
  v = op(v, dpp_u<0x143, 0xc>(id, v));
  return v;
}
__device__ __forceinline__ unsigned lane63_u(unsigned v) {
  return (unsigned)__builtin_amdgcn_readlane((int)v, 63);
}
// inclusive prefix sum over the lanes of the wave
__device__ __forceinline__ unsigned wave_incl_sum_u(unsigned v) {
  return wave_scan_u(v, 0u, [](unsigned x, unsigned y) { return x + y; });
}
__device__ __forceinline__ unsigned wave_min_u(unsigned v) {
  return lane63_u(wave_scan_u(v, 0xffffffffu, [](unsigned x, unsigned y) { return min(x, y); }));
}
__device__ __forceinline__ unsigned wave_max_u(unsigned v) {
  return lane63_u(wave_scan_u(v, 0u, [](unsigned x, unsigned y) { return max(x, y); }));
}
__device__ __forceinline__ unsigned wave_sum_u(unsigned v) { return lane63_u(wave_incl_sum_u(v)); }
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_d(double v) {
  const unsigned long long u = __double_as_longlong(v);
  const unsigned lo = dpp_u<CTRL, ROWS>(0u, (unsigned)u), hi = dpp_u<CTRL, ROWS>(0u, (unsigned)(u >> 32));
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));   // 0 bits = +0.0
}
__device__ __forceinline__ double readlane_d(double v, int l) {
  const unsigned long long u = __double_as_longlong(v);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, l);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), l);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}
// sum over the wave in a fixed order
__device__ __forceinline__ double wave_sum_d(double v) {
  v += dpp_d<0x111, 0xf>(v);
  v += dpp_d<0x112, 0xf>(v);
  v += dpp_d<0x114, 0xf>(v);
  v += dpp_d<0x118, 0xf>(v);
  v += dpp_d<0x142, 0xa>(v);
  v += dpp_d<0x143, 0xc>(v);
  return readlane_d(v, 63);
}

// Block-wide min (OP 0) / max (1) / sum (2) of unsigned values.
template <int OP, int NT>
__device__ __forceinline__ unsigned block_reduce_u(unsigned v, SelSharedT<NT> &ss) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  v = OP == 0 ? wave_min_u(v) : OP == 1 ? wave_max_u(v) : wave_sum_u(v);
  if (lane == 0) ss.red_u[wave] = v;
  lds_barrier();
  if (wave == 0) {
    const unsigned id = OP == 0 ? 0xffffffffu : 0u;
    unsigned x = (lane < NT / 64) ? ss.red_u[lane] : id;
    x = OP == 0 ? wave_min_u(x) : OP == 1 ? wave_max_u(x) : wave_sum_u(x);
    if (lane == 0) ss.bc_u[0] = x;
  }
  lds_barrier();
  const unsigned r = ss.bc_u[0];
  lds_barrier();
  return r;
}

// Sum of four doubles over the block in a fixed order.
template <int NT>
__device__ __forceinline__ void block_sum4_d(double v0, double v1, double v2, double v3, SelSharedT<NT> &ss, double *out) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  v0 = wave_sum_d(v0); v1 = wave_sum_d(v1); v2 = wave_sum_d(v2); v3 = wave_sum_d(v3);
  if (lane == 0) { ss.red_d[0][wave] = v0; ss.red_d[1][wave] = v1; ss.red_d[2][wave] = v2; ss.red_d[3][wave] = v3; }
  lds_barrier();
  if (t < 4) {
    double s = 0.0;
    for (int w = 0; w < NT / 64; ++w) s += ss.red_d[t][w];
    ss.bc_d[t] = s;
  }
  lds_barrier();
  out[0] = ss.bc_d[0]; out[1] = ss.bc_d[1]; out[2] = ss.bc_d[2]; out[3] = ss.bc_d[3];
  lds_barrier();
}

// Scale-matching factor lambda (Eq. lambda_solution) from each thread's
// partial moment sums over the scale-matching set of size M: sum of B - bref,
// of its square, of V - vref and of its square.  The partials go through
// LDS (sc: 4 * NT doubles, one row per sum); wave k < 4 sums row k in a
// fixed order (thread w*64 + lane into lane `lane` for w ascending, then
// across the lanes), and wave 0 forms lambda from the four totals; the
// other waves wait at the barriers rather than each repeat the
// double-precision reduction and arithmetic.  Ends with a barrier; returns
// lambda in every thread.
template <int NT>
__device__ __forceinline__ float block_lambda(double s0, double s1, double s2, double s3, int M,
                                              double bref, float gamma, float eps, float b_floor,
                                              double *sc, SelSharedT<NT> &ss, float *lam_s) {
  static_assert(NT >= 256, "four reducing waves");
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  sc[t] = s0;
  sc[NT + t] = s1;
  sc[2 * NT + t] = s2;
  sc[3 * NT + t] = s3;
  lds_barrier();
  if (wave < 4) {
    const double *row = sc + wave * NT;
    double acc = 0.0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) acc += row[w * 64 + lane];
    acc = wave_sum_d(acc);
    if (lane == 0) ss.bc_d[wave] = acc;
  }
  lds_barrier();
  if (wave == 0) {
    const double a0 = ss.bc_d[0], a1 = ss.bc_d[1], a2 = ss.bc_d[2], a3 = ss.bc_d[3];
    const double mb = a0 / M, mv = a2 / M;
    double vb = a1 / M - mb * mb, vv = a3 / M - mv * mv;
    vb = vb > 0.0 ? vb : 0.0;
    vv = vv > 0.0 ? vv : 0.0;
    // a spread of B within its rounding is none (B equal in exact arithmetic)
    if (sqrt(vb) <= (double)b_floor * (bref + mb)) vb = 0.0;
    if (t == 0) *lam_s = (float)((double)gamma * sqrt(vb) / (sqrt(vv) + (double)eps));
  }
  lds_barrier();
  return *lam_s;
}

// Exclusive prefix sum over threads in index order.
template <int NT>
__device__ __forceinline__ unsigned block_excl_scan_u(unsigned v, SelSharedT<NT> &ss) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const unsigned x = wave_incl_sum_u(v);
  if (lane == 63) ss.red_u[wave] = x;
  lds_barrier();
  unsigned before = 0;
  for (int w = 0; w < wave; ++w) before += ss.red_u[w];
  lds_barrier();
  return before + x - v;
}

constexpr int kCandCap = 1024;   // LDS list of boundary-bin candidates
constexpr int kSegCandCap = 2 * kSegThreads;   // the same in the select kernels of the fused pass

// Boundary search over bin counts held in registers (larger bin = larger
// keys): thread t holds the BPT consecutive bins starting at BPT*t.  For the
// need-th largest counted element, ss.bc_i[0] receives its bin, ss.bc_i[1]
// the count in the bins above it and ss.bc_u[2] the count of its bin;
// ss.bc_u[3] gets the total count.  Ends with a barrier.
template <int BPT, int NT>
__device__ __forceinline__ void bins_boundary(const unsigned *cb, int need, SelSharedT<NT> &ss) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  unsigned c = 0;
#pragma unroll
  for (int q = 0; q < BPT; ++q) c += cb[q];
  const unsigned pre = wave_incl_sum_u(c);
  const unsigned tot = lane63_u(pre);
  unsigned suf = tot - pre + c;        // inclusive suffix sum within the wave
  if (lane == 0) ss.red_u[wave] = tot;
  lds_barrier();
  unsigned higher = 0;                 // counted elements in later waves
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) higher += (w > wave) ? ss.red_u[w] : 0u;
  suf += higher;
  const unsigned above = suf - c;
  if (above < (unsigned)need && (unsigned)need <= suf) {
    unsigned acc = above, bc = 0;
    int bs = BPT * t;
#pragma unroll
    for (int q = BPT - 1; q >= 0; --q) {
      if (acc + cb[q] >= (unsigned)need) { bs = BPT * t + q; bc = cb[q]; break; }
      acc += cb[q];
    }
    ss.bc_i[0] = bs;
    ss.bc_i[1] = (int)acc;
    ss.bc_u[2] = bc;
  }
  if (t == 0) ss.bc_u[3] = suf;
  lds_barrier();
}

// The same over ss.hist (kHistBins bins).
template <int NT>
__device__ __forceinline__ void hist_boundary(int need, SelSharedT<NT> &ss) {
  constexpr int BPT = kHistBins / NT;
  unsigned cb[BPT];
#pragma unroll
  for (int q = 0; q < BPT; ++q) cb[q] = ss.hist[BPT * threadIdx.x + q];
  bins_boundary<BPT, NT>(cb, need, ss);
}

// Compacts the elements j with in(j) into the LDS list (ckey, cpos) in
// (wave, element slot, lane) order, through ballots (no atomics); returns
// nothing, the list length is the caller's count (entries beyond the
// kCandCap slots of the list are dropped).  Ends with a barrier.
template <int PER, int NT, int CAPI = kCandCap, typename InF, typename KeyF, typename PosF>
__device__ __forceinline__ void compact_ballot(InF in, KeyF key, PosF pos, unsigned *ckey, int *cpos,
                                               SelSharedT<NT> &ss) {
  constexpr unsigned CAP = CAPI;
  constexpr int NW = NT / 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  unsigned wc = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) wc += (unsigned)__popcll(__ballot(in(j)));
  if (lane == 0) ss.red_u[wave] = wc;
  lds_barrier();
  unsigned off = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) off += (w < wave) ? ss.red_u[w] : 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const bool i = in(j);
    const uint64_t m = __ballot(i);
    if (i) {
      const unsigned o = off + __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
      if (o < CAP) {
        ckey[o] = key(j);
        cpos[o] = pos(j);
      }
    }
    off += (unsigned)__popcll(m);
  }
  lds_barrier();
}

// The need-th entry (1-based) of C <= NT listed entries under the tie rule
// (key descending, position ascending): xk = its key, pthr = its position.
// Every entry is ranked against all others by tpe consecutive lanes.  Lists
// of NT < C <= 2*NT entries (a boundary bin of exact ties) are ranked two
// entries per thread, each against all others: correct, and slow.
template <int NT>
__device__ __forceinline__ void rank_pick(int C, int need, const unsigned *ckey, const int *cpos,
                                          SelSharedT<NT> &ss, unsigned &xk, int &pthr) {
  const int t = threadIdx.x;
  if (C > NT) {
    const bool two = t + NT < C;
    const unsigned k0 = ckey[t], k1 = two ? ckey[t + NT] : 0u;
    const int p0 = cpos[t], p1 = two ? cpos[t + NT] : 0;
    unsigned r0 = 0, r1 = 0;
    for (int q = 0; q < C; ++q) {
      const unsigned kq = ckey[q];
      const int pq = cpos[q];
      r0 += (kq > k0 || (kq == k0 && pq < p0)) ? 1u : 0u;
      r1 += (kq > k1 || (kq == k1 && pq < p1)) ? 1u : 0u;
    }
    if (r0 == (unsigned)(need - 1)) { ss.bc_u[1] = k0; ss.bc_i[2] = p0; }
    if (two && r1 == (unsigned)(need - 1)) { ss.bc_u[1] = k1; ss.bc_i[2] = p1; }
    lds_barrier();
    xk = ss.bc_u[1];
    pthr = ss.bc_i[2];
    lds_barrier();
    return;
  }
  int tpe = 1;
  while (tpe < 32 && 2 * tpe * C <= NT) tpe *= 2;
  const int q = t / tpe, sub = t & (tpe - 1);
  unsigned rk = 0, kq = 0;
  int pq = 0;
  if (q < C) {
    kq = ckey[q];
    pq = cpos[q];
    // four entries per round, all read before the first compare
    for (int p = sub; p < C; p += 4 * tpe) {
      unsigned kp[4];
      int pp[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = min(p + u * tpe, C - 1);
        kp[u] = ckey[r];
        pp[u] = cpos[r];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        rk += (p + u * tpe < C && (kp[u] > kq || (kp[u] == kq && pp[u] < pq))) ? 1u : 0u;
    }
  }
  if (tpe > 1) rk += swz<1>(rk);
  if (tpe > 2) rk += swz<2>(rk);
  if (tpe > 4) rk += swz<4>(rk);
  if (tpe > 8) rk += swz<8>(rk);
  if (tpe > 16) rk += swz<16>(rk);
  if (q < C && sub == 0 && rk == (unsigned)(need - 1)) {
    ss.bc_u[1] = kq;
    ss.bc_i[2] = pq;
  }
  lds_barrier();
  xk = ss.bc_u[1];
  pthr = ss.bc_i[2];
  lds_barrier();
}

// The need-th entry (1-based) of C <= 2*NT listed entries that share key bits
// 31..18 (one bin of the select histograms), under the tie rule.  Up to
// kRankDirect entries are ranked directly (each against all others, a cost
// that grows with C^2); more are first narrowed to their sub-bin of key bits
// 17..7 by one LDS histogram round, and only that sub-bin is ranked.  The
// list (ckey, cpos) is overwritten.
constexpr int kRankDirect = 192;
template <int NT>
__device__ __forceinline__ void rank_pick_bin(int C, int need, unsigned *ckey, int *cpos,
                                              SelSharedT<NT> &ss, unsigned &xk, int &pthr) {
  if (C <= kRankDirect) {
    rank_pick<NT>(C, need, ckey, cpos, ss, xk, pthr);
    return;
  }
  const int t = threadIdx.x;
  for (int q = t; q < kHistBins; q += NT) ss.hist[q] = 0u;
  unsigned k[2] = {0u, 0u}, sub[2];
  int p[2] = {0, 0};
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    if (t + j * NT < C) {
      k[j] = ckey[t + j * NT];
      p[j] = cpos[t + j * NT];
    }
    sub[j] = (k[j] >> 7) & (unsigned)(kHistBins - 1);
  }
  lds_barrier();
#pragma unroll
  for (int j = 0; j < 2; ++j)
    if (t + j * NT < C) atomicAdd(&ss.hist[sub[j]], 1u);
  lds_barrier();
  hist_boundary<NT>(need, ss);
  const unsigned s2 = (unsigned)ss.bc_i[0];
  const int need2 = need - ss.bc_i[1];
  const int C2 = (int)ss.bc_u[2];
  compact_ballot<2, NT, kSegCandCap>([&](int j) { return t + j * NT < C && sub[j] == s2; },
                                     [&](int j) { return k[j]; }, [&](int j) { return p[j]; },
                                     ckey, cpos, ss);
  rank_pick<NT>(C2, need2, ckey, cpos, ss, xk, pthr);
}

// k-th largest key among the block's non-zero keys (1 <= k <= count), by
// MSB-first 11-bit histogram narrowing of the candidate range over all
// elements.  Returns the key value xk and need = k - #{keys > xk}.
template <int PER, typename KeyF, int NT>
__device__ __forceinline__ void block_select(KeyF key, int k, unsigned &xk, int &need, SelSharedT<NT> &ss) {
  const int t = threadIdx.x;
  unsigned lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const unsigned x = key(j);
    if (x) { lo = min(lo, x); hi = max(hi, x); }
  }
  lo = block_reduce_u<0>(lo, ss);
  hi = block_reduce_u<1>(hi, ss);
  need = k;
  while (lo != hi) {
    const unsigned range = hi - lo;
    const int sh = max(0, 32 - __clz((int)range) - 11);
    for (int q = t; q < kHistBins; q += NT) ss.hist[q] = 0u;
    lds_barrier();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const unsigned x = key(j);
      if (x >= lo && x <= hi) atomicAdd(&ss.hist[(x - lo) >> sh], 1u);
    }
    lds_barrier();
    hist_boundary(need, ss);
    const int bs = ss.bc_i[0];
    need -= ss.bc_i[1];
    const unsigned nlo = lo + ((unsigned)bs << sh);
    const unsigned span = (1u << sh) - 1u;
    const unsigned nhi = (hi - nlo <= span) ? hi : nlo + span;
    lo = nlo;
    hi = nhi;
    lds_barrier();
  }
  xk = lo;
}

constexpr int kEdgeCap = kEdgeEntries;   // LDS tables of E and L corrections next to chunk boundaries

// Exact top-k threshold with the tie rule (key descending, then position
// ascending) over the block's non-zero keys, 1 <= k <= count: element j is
// kept iff key > xk, or key == xk and position <= pthr.
// One histogram pass bins every key over [max(min, max - 8 octaves), max];
// the boundary bin is compacted into an LDS list (ckey, cpos) in a fixed
// order (ballots, no atomics).  A list of at most NT entries is resolved by
// ranking every entry against all others under the tie rule; a longer one by
// 11-bit histogram rounds.  When the boundary falls below the binned range or
// its bin overflows the list, full-range narrowing over all elements is used.
// Ends with a barrier.
template <int PER, typename KeyF, typename PosF, int NT>
__device__ __forceinline__ void block_threshold(KeyF key, PosF pos, int k, unsigned &xk, int &pthr,
                                                SelSharedT<NT> &ss, unsigned *ckey, int *cpos) {
  constexpr int NW = NT / 64;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  // the range reduction's barrier also orders this clear before the binning
  for (int q = t; q < kHistBins; q += NT) ss.hist[q] = 0u;
  unsigned lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const unsigned x = key(j);
    if (x) { lo = min(lo, x); hi = max(hi, x); }
  }
  lo = wave_min_u(lo);
  hi = wave_max_u(hi);
  if (lane == 0) { ss.red_u[wave] = lo; ss.red_u2[wave] = hi; }
  lds_barrier();
  lo = 0xffffffffu;
  hi = 0u;
#pragma unroll
  for (int w = 0; w < NW; ++w) { lo = min(lo, ss.red_u[w]); hi = max(hi, ss.red_u2[w]); }
  if (hi - lo > (8u << 23)) lo = hi - (8u << 23);      // at most 8 octaves below the max
  const int sh0 = max(0, 32 - __clz((int)(hi - lo)) - 11);
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const unsigned x = key(j);
    if (x >= lo && hi >= lo) atomicAdd(&ss.hist[(x - lo) >> sh0], 1u);
  }
  lds_barrier();
  hist_boundary(k, ss);
  const unsigned counted = ss.bc_u[3];
  bool fallback = counted < (unsigned)k;                // boundary below the binned range
  unsigned b0 = 0, C = 0;
  int need = k;
  if (!fallback) {
    b0 = (unsigned)ss.bc_i[0];
    need = k - ss.bc_i[1];
    C = ss.hist[b0];
    fallback = C > (unsigned)kCandCap;
  }
  lds_barrier();
  if (fallback) {
    int nd;
    block_select<PER>(key, k, xk, nd, ss);
    unsigned eq = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) eq += key(j) == xk;
    if (block_reduce_u<2>(eq, ss) == (unsigned)nd) {
      pthr = 0x7fffffff;
    } else {
      auto pkey = [&](int j) -> unsigned { return key(j) == xk ? 0xffffffffu - (unsigned)pos(j) : 0u; };
      unsigned xp;
      int n2;
      block_select<PER>(pkey, nd, xp, n2, ss);
      pthr = (int)(0xffffffffu - xp);
    }
    return;
  }
  // compact the boundary bin in (wave, element slot, lane) order
  compact_ballot<PER, NT>([&](int j) { const unsigned x = key(j); return x >= lo && ((x - lo) >> sh0) == b0; },
                          key, pos, ckey, cpos, ss);
  if (C <= (unsigned)NT) {
    rank_pick<NT>((int)C, need, ckey, cpos, ss, xk, pthr);
    return;
  }
  // resolve the key inside the bin: 11 bits at a time from bit sh0 down
  const unsigned blo = lo + (b0 << sh0);                // smallest key of the bin
  unsigned pre = 0, pmask = 0;                          // known bits of (x - blo)
  int sh = sh0;
  unsigned E = C;                                       // candidates matching the prefix
  while (sh > 0) {
    const int nb = min(sh, 11);
    sh -= nb;
    const unsigned bm = (1u << nb) - 1u;
    for (int q = t; q < kHistBins; q += NT) ss.hist[q] = 0u;
    lds_barrier();
    for (int q = t; q < (int)C; q += NT) {
      const unsigned d = ckey[q] - blo;
      if ((d & pmask) == pre) atomicAdd(&ss.hist[(d >> sh) & bm], 1u);
    }
    lds_barrier();
    hist_boundary(need, ss);
    const unsigned bl = (unsigned)ss.bc_i[0];
    need -= ss.bc_i[1];
    E = ss.hist[bl];
    pre |= bl << sh;
    pmask |= bm << sh;
    lds_barrier();
  }
  xk = blo + pre;
  if (E == (unsigned)need) {
    pthr = 0x7fffffff;
    return;
  }
  // the `need` lowest positions among the E ties (positions < 2^15)
  unsigned ppre = 0, ppm = 0;
  for (int ps = 15; ps > 0;) {
    const int nb = min(ps, 11);
    ps -= nb;
    const unsigned bm = (1u << nb) - 1u;
    for (int q = t; q < kHistBins; q += NT) ss.hist[q] = 0u;
    lds_barrier();
    for (int q = t; q < (int)C; q += NT) {
      if (ckey[q] != xk) continue;
      const unsigned d = 0x7fffu - (unsigned)cpos[q];   // larger d = lower position
      if ((d & ppm) == ppre) atomicAdd(&ss.hist[(d >> ps) & bm], 1u);
    }
    lds_barrier();
    hist_boundary(need, ss);
    const unsigned bl = (unsigned)ss.bc_i[0];
    need -= ss.bc_i[1];
    ppre |= bl << ps;
    ppm |= bm << ps;
    lds_barrier();
  }
  pthr = (int)(0x7fffu - ppre);
}

using SelShared = SelSharedT<kSelThreads>;

// ---------------------------------------------------------------- select kernel
// LDS: S padded by one word per kSelPer (thread-contiguous reads hit distinct
// banks), reused as the slot table.
__device__ __forceinline__ int pad32(int i) { return i + i / kSelPer; }
constexpr int kArrWords = kMaxSelLen + kMaxSelLen / kSelPer + 64;

template <int MODE>
__global__ __launch_bounds__(kSelThreads) void k_select(SelArgs a, SeqTable st) {
  constexpr int PER = kSelPer;
  extern __shared__ __align__(16) float arr[];
  __shared__ SelShared ss;
  const int b = blockIdx.x, h = blockIdx.y, t = threadIdx.x;
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;                           // candidate set [0, nc)
  const int K = head_budget(st, a.hb, a.Hkv, b, h);
  const int64_t base = (int64_t)h * a.T + st.cu[b];
  // LDS: arr [pad32 extent of kMaxSelLen], candidate list, then per-mode tables
  unsigned *ckey = reinterpret_cast<unsigned *>(arr + kArrWords);
  int *cpos = reinterpret_cast<int *>(ckey + kCandCap);

  if constexpr (MODE != SEL_TOPK) {
    // The L neighbours of positions next to a chunk boundary of vec_VP that lie
    // in the neighbouring chunk.  Boundary c*CH (c >= 1) covers the 2r
    // positions [c*CH - r, c*CH + r); the host keeps nbnd*2r <= kEdgeCap.
    const int r = a.radius, CH = a.vp_chunk;
    const bool use_l = (a.terms & 2u) != 0;
    const int nbnd = (use_l && CH < n) ? (n - 1) / CH : 0;      // boundaries inside the sequence
    const int nedge = nbnd * 2 * r;
    float *edge = reinterpret_cast<float *>(cpos + kCandCap);     // E at those positions
    float *fixt = edge + kEdgeCap;                                // their L correction
    const float *re = a.ring + a.ring_slot * a.ring_stride + base;   // E of this layer
    for (int q = t; q < nedge; q += kSelThreads) {
      const int c = q / (2 * r) + 1, o = q - (c - 1) * 2 * r;
      const int u = c * CH - r + o;
      const float e = re[min(max(u, 0), n - 1)];
      edge[q] = (u >= 0 && u < n) ? e : 0.f;
    }
    lds_barrier();
    for (int q = t; q < nedge; q += kSelThreads) {
      const int c = q / (2 * r) + 1, o = q - (c - 1) * 2 * r;
      const int i = c * CH - r + o;                 // position next to boundary c*CH
      const int lo = max(0, i - r), hi = min(n - 1, i + r);
      float sum = 0.f;
      if (i < c * CH) {                             // left of the boundary: right neighbours
        for (int u = c * CH; u <= hi; ++u) sum += edge[(c - 1) * 2 * r + (u - (c * CH - r))];
      } else {                                      // right of it: left neighbours
        for (int u = lo; u < c * CH; ++u) sum += edge[(c - 1) * 2 * r + (u - (c * CH - r))];
      }
      fixt[q] = (i >= 0 && i < n) ? sum / (float)(hi - lo + 1) : 0.f;
    }
    // correction of position i (0 when i is not next to a boundary)
    auto vfix = [&](int i) -> float {
      if (nbnd == 0) return 0.f;
      const int c = (i + r) / CH;
      const int o = i - (c * CH - r);
      return (c >= 1 && c <= nbnd && o < 2 * r) ? fixt[(c - 1) * 2 * r + o] : 0.f;
    };
    // B into LDS (strided: element j of thread t is position t + j*kSelThreads);
    // all loads of the phase are issued before any is used.
    {
      const int tt = opaque(t);   // keeps the phase's address arithmetic local
      const float *pb = a.vec_B + base;
      float bv[PER];
#pragma unroll
      for (int j = 0; j < PER; ++j) bv[j] = pb[min(tt + j * kSelThreads, n - 1)];
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (tt + j * kSelThreads < n) arr[pad32(tt + j * kSelThreads)] = bv[j];
    }
    lds_barrier();
    // Scale-matching set: top M = min(rho K, |I|) of B over I (Eq. scale_matching_set).
    int M = scale_set_size(a.rho, K);
    if (M > nc) M = nc;
    if (M < 0) M = 0;
    const bool calib = M > 0 && a.use_last_query;
    uint64_t msk = 0;
    if (calib) {
      auto keyB = [&](int j) -> unsigned {
        const int i = t + j * kSelThreads;
        const unsigned kx = float_key(arr[pad32(i)]);   // i < kMaxSelLen: inside arr
        return i < nc ? kx : 0u;
      };
      auto posf = [&](int j) -> int { return t + j * kSelThreads; };
      if (M >= nc) {
#pragma unroll
        for (int j = 0; j < PER; ++j) msk |= (uint64_t)(t + j * kSelThreads < nc ? 1u : 0u) << j;
      } else {
        unsigned xm;
        int pm;
        block_threshold<PER>(keyB, posf, M, xm, pm, ss, ckey, cpos);
#pragma unroll
        for (int j = 0; j < PER; ++j) {
          const unsigned kj = keyB(j);
          msk |= (uint64_t)(kj > xm || (kj == xm && posf(j) <= pm) ? 1u : 0u) << j;
        }
      }
    }
    // V for the thread's positions: vec_VP, completed next to chunk boundaries.
    const int tt = opaque(t);
    float vp[PER];
    {
      const float *pv = a.vec_VP + base;
#pragma unroll
      for (int j = 0; j < PER; ++j) vp[j] = pv[min(tt + j * kSelThreads, n - 1)];
#pragma unroll
      for (int j = 0; j < PER; ++j) vp[j] += vfix(tt + j * kSelThreads);
    }
    float lam = 0.f;
    if (calib) {
      // population moments over the set in double; B shifted by the set minimum
      float bv[PER];
#pragma unroll
      for (int j = 0; j < PER; ++j) bv[j] = arr[pad32(tt + j * kSelThreads)];
      unsigned kmin = 0xffffffffu;
#pragma unroll
      for (int j = 0; j < PER; ++j)
        kmin = ((msk >> j) & 1ull) ? min(kmin, float_key(bv[j])) : kmin;
      kmin = block_reduce_u<0>(kmin, ss);
      const double bref = (double)key_float(kmin);
      // V is shifted by the smallest V of the set as well: the variance is
      // the same, and a set of equal V gives exactly 0
      unsigned vmin = 0xffffffffu;
#pragma unroll
      for (int j = 0; j < PER; ++j)
        vmin = ((msk >> j) & 1ull) ? min(vmin, float_key(vp[j])) : vmin;
      vmin = block_reduce_u<0>(vmin, ss);
      const double vref = (double)key_float(vmin);
      double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const bool in = (msk >> j) & 1ull;
        const double db = in ? (double)bv[j] - bref : 0.0, dv = in ? (double)vp[j] - vref : 0.0;
        s0 += db; s1 += db * db; s2 += dv; s3 += dv * dv;
      }
      double sums[4];
      block_sum4_d(s0, s1, s2, s3, ss, sums);
      const double mb = sums[0] / M, mv = sums[2] / M;
      double vb = sums[1] / M - mb * mb, vv = sums[3] / M - mv * mv;
      vb = vb > 0.0 ? vb : 0.0;
      vv = vv > 0.0 ? vv : 0.0;
      lam = (float)((double)a.gamma * sqrt(vb) / (sqrt(vv) + (double)a.eps));   // Eq. lambda_solution
    }
    if (t == 0) {
      a.lambda_ws[b * a.Hkv + h] = lam;
      if (a.out_lambda) a.out_lambda[b * a.Hkv + h] = lam;
    }
    // S = B + lambda V (Eq. bacon_score), in place of B; each thread touches
    // only its own positions.
    // With pooling before calibration the candidates get pool(B) + lambda V
    // instead, the score the top-K then ranks unpooled.
    const bool mean_b = a.pool_mode == POOL_MEAN_B;
    const int hp = a.pool_half;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int i = tt + j * kSelThreads;
      if (i < n) {
        float bi = arr[pad32(i)];
        if (mean_b && i < nc) {
          const int lo = max(0, i - hp), hi = min(nc - 1, i + hp);
          double acc = 0.0;
          for (int u = lo; u <= hi; ++u) acc += (double)arr[pad32(u)];
          bi = (float)(acc / (double)(hi - lo + 1));
        }
        a.out_S[base + i] = fmaf(lam, vp[j], bi);
        if (a.out_V) a.out_V[base + i] = vp[j];
        if (a.out_E) a.out_E[base + i] = re[i];
      }
    }
    return;
  } else {
    float sv[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) sv[j] = a.in_S[base + min(t + j * kSelThreads, n - 1)];
#pragma unroll
    for (int j = 0; j < PER; ++j)
      if (t + j * kSelThreads < nc) arr[pad32(t + j * kSelThreads)] = sv[j];
  }
  lds_barrier();

  // Pooled score over I and its keys, contiguous ownership: positions
  // [t*PER, t*PER + PER).  The mean pool slides window sums in double; the
  // max pool scans each window; with pooling before calibration S is taken
  // as it is.
  const int i0 = t * PER;
  unsigned key[PER];
  {
    const int hp = a.pool_half;
#pragma unroll
    for (int j = 0; j < PER; ++j) key[j] = 0u;
    if (i0 < nc && a.pool_mode == POOL_MEAN_B) {
#pragma unroll
      for (int j = 0; j < PER; ++j)
        if (i0 + j < nc) key[j] = float_key(arr[pad32(i0 + j)]);
    } else if (i0 < nc && a.pool_mode == POOL_MAX_S) {
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int i = i0 + j;
        if (i < nc) {
          const int lo = max(0, i - hp), hi = min(nc - 1, i + hp);
          float mx = arr[pad32(lo)];
          for (int u = lo + 1; u <= hi; ++u) mx = fmaxf(mx, arr[pad32(u)]);
          key[j] = float_key(mx);
        }
      }
    } else if (i0 < nc) {
      int lo = max(0, i0 - hp), hi = min(nc - 1, i0 + hp);
      double acc = 0.0;
      for (int u = lo; u <= hi; ++u) acc += (double)arr[pad32(u)];
      const double inv_full = 1.0 / (double)(2 * hp + 1);
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int i = i0 + j;
        // both reads are unconditional (clamped) so they never wait on a branch
        const float in_v = arr[pad32(min(i + 1 + hp, nc - 1))];
        const float out_v = arr[pad32(max(i - hp, 0))];
        if (i < nc) {
          const int cnt = hi - lo + 1;
          double inv = inv_full;
          if (cnt != 2 * hp + 1) inv = 1.0 / (double)cnt;
          key[j] = float_key((float)(acc * inv));
          acc += (i + 1 + hp <= nc - 1) ? (double)in_v : 0.0;
          acc -= (i - hp >= 0) ? (double)out_v : 0.0;
          lo = max(0, i + 1 - hp);
          hi = min(nc - 1, i + 1 + hp);
        }
      }
    }
  }
  lds_barrier();   // pooled values read; arr is reused as the slot table

  // Top-K over I (Eq. topk_selection), emitted in ascending position.
  const int kept = min(K, nc);
  uint64_t msk = 0;
  if (kept == nc) {
#pragma unroll
    for (int j = 0; j < PER; ++j) msk |= (uint64_t)(i0 + j < nc ? 1u : 0u) << j;
  } else if (kept > 0) {
    auto keyS = [&](int j) -> unsigned { return key[j]; };
    auto posf = [&](int j) -> int { return i0 + j; };
    unsigned xk;
    int pk;
    block_threshold<PER>(keyS, posf, kept, xk, pk, ss, ckey, cpos);
#pragma unroll
    for (int j = 0; j < PER; ++j)
      msk |= (uint64_t)(key[j] > xk || (key[j] == xk && i0 + j <= pk) ? 1u : 0u) << j;
  }
  int32_t *idx = a.idx + head_idx_base(st, a.hb, a.Hkv, b, h);
  int *tbl = reinterpret_cast<int *>(arr);
  unsigned slot = block_excl_scan_u((unsigned)__popcll(msk), ss);
  {
    uint64_t m2 = msk;
    while (m2) {
      const int j = __builtin_ctzll(m2);
      m2 &= m2 - 1;
      idx[slot] = i0 + j;
      tbl[slot] = i0 + j;
      ++slot;
    }
  }
  for (int j = kept + t; j < K; j += kSelThreads) idx[j] = -1;

}

size_t select_lds_bytes(int mode, int max_len) {
  (void)max_len;   // arr always spans kMaxSelLen so strided reads need no clamping
  size_t bytes = (size_t)kArrWords * sizeof(float) +                              // arr (padded)
                 2 * kCandCap * sizeof(unsigned);                                // candidate list
  if (mode != SEL_TOPK) bytes += 2 * kEdgeCap * sizeof(float);                   // boundary tables
  return bytes + sizeof(SelShared);
}

hipError_t launch_select(int mode, int max_len, const SelArgs &a, const SeqTable &st,
                         hipStream_t s) {
  dim3 grid(st.batch, a.Hkv), block(kSelThreads);
  const size_t lds = select_lds_bytes(mode, max_len) - sizeof(SelShared);
  if (lds + sizeof(SelShared) > kLdsBytes) return hipErrorInvalidValue;
  if (mode == SEL_CALIB) {
    allow_lds(k_select<SEL_CALIB>, lds);
    hipLaunchKernelGGL((k_select<SEL_CALIB>), grid, block, lds, s, a, st);
  } else {
    allow_lds(k_select<SEL_TOPK>, lds);
    hipLaunchKernelGGL((k_select<SEL_TOPK>), grid, block, lds, s, a, st);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------- histogram select
// Four kernels after the fused pass; none waits on another workgroup.  The
// selections use per-(sequence, KV head) histograms of the order-preserving
// keys of the scores (kHBins bins, 32 per octave of a float): one kernel
// accumulates a histogram, the next finds the boundary bin of its top-k in
// one scan of the bins.  Work on positions stays spread over the segments of
// kSegLen positions (two positions per thread); the segments exchange only
// their lists of entries at or above the boundary bin, and the exact order
// inside the boundary bin (ties to the lower position) is resolved on those
// short lists.  Lists longer than one workgroup holds fall back to the exact
// block select over the whole sequence.
//
//  * segment_calib (one workgroup per segment and KV head): forms
//    L = P_r E from the history and V = E + L + T (Eq. structurally_calibrated_evidence),
//    writes the pooled B and V over I, finds the boundary bin of the top-M of
//    B in the B histogram the fused pass accumulated (Eqs. scale_matching_size,
//    scale_matching_set), and lists its candidates at or above it with their V.
//  * segment_score (same grid): every workgroup of a (sequence, KV head)
//    resolves the scale-matching set from the segments' lists and solves
//    lambda (Eq. lambda_solution) -- the same exact computation in each, so no
//    workgroup waits for another -- then forms the pooled score
//    pB + lambda pV of its segment (Eq. bacon_score, pooled) and adds its keys
//    to the S histogram.
//  * segment_cand (same grid): the boundary bin of the top-K of the pooled
//    score (Eq. topk_selection) and the segment's list of entries at or above it.
//  * final_topk (`parts` workgroups per (sequence, KV head)): the top-K from
//    the lists, the kept positions in ascending order, and each workgroup's
//    share of the compacted cache rows.
// Boundary bins of up to kSegCandCap entries are resolved on the lists
// (large ones narrowed to a sub-bin first).  In a prompt call the four run
// as two launches per layer that also carry the previous and next layers'
// work (k_sel_a, k_sel_b).
constexpr int kSegPer = kSegLen / kSegThreads;             // positions per thread (strided)
constexpr int kSegWin = kSegLen + 2 * kPoolHalo;           // segment plus pool halo
constexpr int kSegWinJ = (kSegWin + kSegThreads - 1) / kSegThreads;
constexpr int kMaxRadius = 16;                             // largest coherence radius
constexpr int kSegE = kSegWin + 2 * kMaxRadius;            // E over the window and the radius
constexpr int kSegEJ = (kSegE + kSegThreads - 1) / kSegThreads;
constexpr int kAllPer = kMaxSelLen / kSegThreads;          // positions per thread of the register fallback
constexpr int kHPer = kHBins / kSegThreads;                // histogram bins per thread
constexpr int kListPer = 4;                                // list entries per thread
constexpr int kListSpec = 2;                               // of them loaded before the counts are known
constexpr int kListCap = kListPer * kSegThreads;           // list entries of a (sequence, KV head)
constexpr int kMaxSegs = kMaxSeqLen / kSegLen;             // segments of a sequence
constexpr int kMomChunk = 4096;                            // scale-matching entries per LDS round
static_assert(kAllPer <= 32 && kHPer % 4 == 0 && kMaxSegs <= 64, "select layout");

// Budget fields of the select kernels.  The sequence table sits in the
// kernel arguments, the optional per-sequence (sb) and per-head (hb) tables
// in global memory; read through one conditional expression, the two are
// merged into a generic load of a selected pointer, whose wait also waits
// for every global load the wave has in flight.  The kernel-argument word is
// taken apart (a scalar load behind an empty asm), and a table only when it
// is given, waited for inside its branch: where no table is given, no wait
// for global loads follows.
__device__ __forceinline__ int kern_word(const int32_t &w) {
  // (uniform: the read-first-lane is free, and lets the scalar constraint
  // hold wherever the compiler placed the load)
  int v = __builtin_amdgcn_readfirstlane(w);
  asm volatile("" : "+s"(v));
  return v;
}
__device__ __forceinline__ int table_word(const int *p) {
  int v = *p;
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ int sel_seq_budget(const SeqTable &st, const int4 *sb, int b) {
  int v = kern_word(st.budget[b]);
  if (sb) v = table_word(&sb[b].x);
  return v;
}
__device__ __forceinline__ int sel_seq_kept_base(const SeqTable &st, const int4 *sb, int b) {
  int v = kern_word(st.kept_base[b]);
  if (sb) v = table_word(&sb[b].z);
  return v;
}
__device__ __forceinline__ int sel_head_budget(const SeqTable &st, const int2 *hb, int Hkv, int b, int h,
                                               const int4 *sb) {
  int v = sel_seq_budget(st, sb, b);
  if (hb) v = table_word(&hb[b * Hkv + h].x);
  return v;
}
__device__ __forceinline__ int64_t sel_head_idx_base(const SeqTable &st, const int2 *hb, int Hkv, int b,
                                                     int h, const int4 *sb) {
  int v = kern_word(st.idx_base[b]);
  if (sb) v = table_word(&sb[b].y);
  int w;
  if (hb) w = table_word(&hb[b * Hkv + h].y);
  else w = h * sel_seq_budget(st, sb, b);
  return (int64_t)v + w;
}

__device__ __forceinline__ int find_seg(const SeqTable &st, int seg) {
  int b = 0;
  while (b + 1 < st.batch && st.seg_base[b + 1] <= seg) ++b;
  return b;
}

// Slots of the set elements of a strided layout (element j of thread t is
// item t + j*NT) in item order: pre[j*NW + wave] receives the number of set
// elements before (j, wave), and pre[PER*NW] the total; an element's slot is
// pre[j*NW + wave] plus its lane rank in the ballot.  Ends with a barrier.
template <int PER, int NT>
__device__ __forceinline__ void ordered_bases(uint32_t msk, unsigned *pre) {
  constexpr int NW = NT / 64, NE = PER * NW, E = (NE + 63) / 64;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const uint64_t m = __ballot((msk >> j) & 1u);
    if (lane == 0) pre[j * NW + wave] = (unsigned)__popcll(m);
  }
  lds_barrier();
  if (wave == 0) {
    unsigned x[E], s = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      x[e] = (lane * E + e < NE) ? pre[lane * E + e] : 0u;
      s += x[e];
    }
    const unsigned incl = wave_incl_sum_u(s);
    unsigned ex = incl - s;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (lane * E + e < NE) pre[lane * E + e] = ex;
      ex += x[e];
    }
    if (lane == 63) pre[NE] = incl;
  }
  lds_barrier();
}
__device__ __forceinline__ unsigned lane_rank(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

// The thread's kHPer consecutive bins of a histogram row, summed over
// `copies` consecutive copies of the row.
template <int COPIES = 1>
__device__ __forceinline__ void load_bins(const unsigned *gh, unsigned *cb) {
  u32x4 v[COPIES][kHPer / 4];
#pragma unroll
  for (int c = 0; c < COPIES; ++c) {
    const u32x4 *hp = reinterpret_cast<const u32x4 *>(gh + (int64_t)c * kHBins + kHPer * threadIdx.x);
#pragma unroll
    for (int q = 0; q < kHPer / 4; ++q) v[c][q] = hp[q];
  }
#pragma unroll
  for (int q = 0; q < kHPer / 4; ++q) {
    u32x4 x = v[0][q];
#pragma unroll
    for (int c = 1; c < COPIES; ++c) x += v[c][q];
    cb[4 * q + 0] = x.x; cb[4 * q + 1] = x.y; cb[4 * q + 2] = x.z; cb[4 * q + 3] = x.w;
  }
}

// Exact top-k threshold (xk, pthr) of the keys key(j), j < PER, of the block
// (0 = not a candidate) from the histogram gh of those keys: element j is
// kept iff key > xk, or key == xk and position <= pthr.  1 <= k <= count.
// Ends with a barrier.
template <int PER, int COPIES, typename KeyF, typename PosF>
__device__ __forceinline__ void hist_threshold(const unsigned *gh, KeyF key, PosF pos, int k,
                                               unsigned &xk, int &pthr,
                                               SelSharedT<kSegThreads> &ss, unsigned *ckey,
                                               int *cpos) {
  constexpr int NT = kSegThreads;
  unsigned cb[kHPer];
  load_bins<COPIES>(gh, cb);
  bins_boundary<kHPer, NT>(cb, k, ss);
  const int beta = ss.bc_i[0];
  const int need = k - ss.bc_i[1];
  const unsigned C = ss.bc_u[2];
  lds_barrier();
  if (C <= (unsigned)kCandCap) {
    compact_ballot<PER, NT>([&](int j) { const unsigned x = key(j); return x != 0u && hbin(x) == beta; },
                            key, pos, ckey, cpos, ss);
    rank_pick_bin<NT>((int)C, need, ckey, cpos, ss, xk, pthr);
  } else {
    block_threshold<PER>(key, pos, k, xk, pthr, ss, ckey, cpos);
  }
}

// Exact top-k threshold (xk, pthr) over the positions [0, n) of a sequence
// longer than the register form holds (n > kAllPer * NT), its keys read from
// global memory once per step: the boundary bin from the histogram gh (key
// bits 30..18; the method's scores are non-negative, so bit 31 is set), then
// LDS histograms of bits 17..7 and 6..0 of the keys inside it, then the
// position of the need-th key equal to the threshold (position ascending)
// from counts over contiguous ranges of positions.  Kept iff key > xk, or
// key == xk and position <= pthr.  1 <= k <= the count of nonzero keys.
// keyf(i) is the key of position i (0: not a candidate).  Ends with a barrier.
template <int COPIES, typename KeyF>
__device__ __forceinline__ void stream_threshold(const unsigned *gh, KeyF keyf, int n, int k,
                                                 unsigned &xk, int &pthr,
                                                 SelSharedT<kSegThreads> &ss) {
  constexpr int NT = kSegThreads;
  const int t = threadIdx.x;
  unsigned cb[kHPer];
  load_bins<COPIES>(gh, cb);
  bins_boundary<kHPer, NT>(cb, k, ss);
  const unsigned beta = (unsigned)ss.bc_i[0];
  int need = k - ss.bc_i[1];
  lds_barrier();
  unsigned digit[2];
#pragma unroll
  for (int lev = 0; lev < 2; ++lev) {
    for (int q = t; q < kHistBins; q += NT) ss.hist[q] = 0u;
    lds_barrier();
    for (int i = t; i < n; i += NT) {
      const unsigned x = keyf(i);
      if (x == 0u || (unsigned)hbin(x) != beta) continue;
      if (lev == 0) {
        atomicAdd(&ss.hist[(x >> 7) & (kHistBins - 1)], 1u);
      } else if (((x >> 7) & (kHistBins - 1)) == digit[0]) {
        atomicAdd(&ss.hist[x & 127u], 1u);
      }
    }
    lds_barrier();
    hist_boundary<NT>(need, ss);
    digit[lev] = (unsigned)ss.bc_i[0];
    need -= ss.bc_i[1];
    lds_barrier();
  }
  xk = 0x80000000u | (beta << 18) | (digit[0] << 7) | digit[1];
  // the need-th position (ascending) among the keys equal to xk
  const int ch = (n + NT - 1) / NT;
  const int i0 = min(n, t * ch), i1 = min(n, i0 + ch);
  if (t == 0) ss.bc_i[2] = n - 1;   // in range whatever the counts say
  unsigned c = 0;
  for (int i = i0; i < i1; ++i) c += keyf(i) == xk ? 1u : 0u;
  const unsigned ex = block_excl_scan_u<NT>(c, ss);
  if (ex < (unsigned)need && (unsigned)need <= ex + c) {
    unsigned r = ex;
    for (int i = i0; i < i1; ++i)
      if (keyf(i) == xk && ++r == (unsigned)need) {
        ss.bc_i[2] = i;
        break;
      }
  }
  lds_barrier();
  pthr = ss.bc_i[2];
  lds_barrier();
}

// The lists of the nseg segments of a (sequence, KV head) as one sequence of
// entries e = t + j*NT: segment e / cap, slot e % cap.  `fits` is false when
// a segment's count exceeds cap.
struct ListView {
  int nseg, cap;
  bool fits;
};

// Calibration kernel (segment_calib).
__device__ __forceinline__ void segcal_body(const SegArgs &a, const SeqTable &st, int gs, int h, int b) {
  constexpr int NT = kSegThreads, PER = kSegPer, NW = NT / 64;
  // zeroed slots past the end of the LDS windows: the neighbourhood sums of
  // the last window positions read E up to two slots past its window (at
  // the largest radius)
  constexpr int TAPS = 8;
  __shared__ float Bs[kSegWin + TAPS], Vs[kSegWin + TAPS];
  __shared__ float Es[kSegE + TAPS];
  __shared__ SelSharedT<NT> ss;
  __shared__ unsigned pre[PER * NW + 1];
  const int t = threadIdx.x;
  const int wave = t >> 6;
  const int sg = gs - st.seg_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int i0 = sg * kSegLen;
  const int w0 = i0 - kPoolHalo;                    // position of Bs[0]
  const int64_t base = (int64_t)h * a.T + st.cu[b];
  const int r = a.radius;
  const bool use_l = (a.terms & 2u) != 0;
  int M = scale_set_size(a.rho, sel_head_budget(st, a.hb, a.Hkv, b, h, a.sb));
  M = max(0, min(M, nc));
  const bool calib = M > 0 && a.use_last_query;
  // the bins of the B histogram (accumulated by the fused pass, in kHCopies
  // copies): loaded raw and summed once the window loads below are in flight
  u32x4 hv[kHCopies][kHPer / 4];
  {
    const unsigned *gh = a.hist_B + ((int64_t)b * a.Hkv + h) * kHCopies * kHBins;
#pragma unroll
    for (int c = 0; c < kHCopies; ++c)
#pragma unroll
      for (int q = 0; q < kHPer / 4; ++q)
        hv[c][q] = reinterpret_cast<const u32x4 *>(gh + (int64_t)c * kHBins + kHPer * t)[q];
  }
  const float *re = a.ring + a.ring_slot * a.ring_stride + base;   // E of this layer
  {
    // clear this segment's slice of the S histogram that the score kernel
    // accumulates next (its readers of the previous layer are done)
    const int nseg = st.seg_base[b + 1] - st.seg_base[b];
    const int sl = 4 * ((kHBins / 4 + nseg - 1) / nseg);
    unsigned *hs = a.hist_S + ((int64_t)b * a.Hkv + h) * kHBins;
    for (int q = sg * sl + 4 * t; q < min(kHBins, (sg + 1) * sl); q += 4 * NT)
      *reinterpret_cast<u32x4 *>(hs + q) = u32x4{0u, 0u, 0u, 0u};
  }

  // one round of loads: B and T (the earlier layers' E, oldest first) over
  // the window, E over the window widened by the coherence radius
  {
    const int tt = opaque(t);
    float bv[kSegWinJ], tv[kSegWinJ], ev[kSegEJ];
#pragma unroll
    for (int j = 0; j < kSegWinJ; ++j) {
      const int u = min(max(w0 + tt + j * NT, 0), n - 1);
      bv[j] = a.vec_B[base + u];
      tv[j] = 0.f;
    }
#pragma unroll
    for (int j = 0; j < kSegEJ; ++j) {
      const int u = min(max(w0 - kMaxRadius + tt + j * NT, 0), n - 1);
      ev[j] = re[u];
    }
    const bool use_t = (a.terms & 4u) && a.ring_cnt > 0;
    if (use_t) {
      // four earlier layers per round, all loads of a round in flight; past
      // the oldest layer the slot index repeats (an L2 hit) and is not added
      for (int l0 = 0; l0 < a.ring_cnt; l0 += 4) {
        float x[4][kSegWinJ];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int l = max(a.ring_cnt - l0 - i, 1);       // oldest first
          const float *rt = a.ring + ((a.ring_slot - l + a.ring_slots) % a.ring_slots) * a.ring_stride + base;
#pragma unroll
          for (int j = 0; j < kSegWinJ; ++j) x[i][j] = rt[min(max(w0 + tt + j * NT, 0), n - 1)];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < kSegWinJ; ++j) tv[j] += (l0 + i < a.ring_cnt) ? x[i][j] : 0.f;
      }
    }
    // E is 0 outside the sequence in LDS, so that a neighbourhood sum needs
    // no per-position bounds
#pragma unroll
    for (int j = 0; j < kSegEJ; ++j) {
      const int u = w0 - kMaxRadius + tt + j * NT;
      if (tt + j * NT < kSegE) Es[tt + j * NT] = (u >= 0 && u < n) ? ev[j] : 0.f;
    }
    if (t < TAPS) Es[kSegE + t] = 0.f;
    lds_barrier();
    // V = E + L + T (Eq. structurally_calibrated_evidence, per the terms
    // mask), L = P_r E over the sequence-truncated neighbourhood
    // (Eq. intra_layer_coherence), T the mean of the earlier layers' E
    // (Eq. inter_layer_persistence).  The neighbourhood sums are taken for
    // three consecutive window positions per thread, whose 2r + 1 taps
    // overlap (2r + 3 LDS reads instead of 3 (2r + 1)), each summed in
    // position order (a tap outside the sequence adds 0), and pass through
    // Vs to the layout of the loads.
    if (use_l) {
      const int q0 = 3 * t;
      if (q0 < kSegWin) {
        const float *ep = Es + q0 + kMaxRadius - r;   // ep[k]: tap k of position q0 (k <= 2r)
        float s0, s1, s2;
        if (r == 0) {
          s0 = ep[0]; s1 = ep[1]; s2 = ep[2];
        } else {
          s0 = ep[0];
          s1 = ep[1];
          s0 += s1;
          s2 = 0.f;
#pragma unroll 4
          for (int k = 2; k <= 2 * r; ++k) {
            const float x = ep[k];
            s0 += x; s1 += x; s2 += x;
          }
          const float x = ep[2 * r + 1];
          s1 += x;
          s2 += x;
          s2 += ep[2 * r + 2];
        }
        Vs[q0] = s0;
        if (q0 + 1 < kSegWin) Vs[q0 + 1] = s1;
        if (q0 + 2 < kSegWin) Vs[q0 + 2] = s2;
      }
      lds_barrier();
    }
    const float inv_cnt = a.ring_cnt ? 1.f / (float)a.ring_cnt : 0.f;
#pragma unroll
    for (int j = 0; j < kSegWinJ; ++j) {
      const int q = tt + j * NT;
      if (q < kSegWin) {
        const int u = w0 + q;
        float v = ((a.terms & 1u) ? Es[q + kMaxRadius] : 0.f) + (use_t ? tv[j] * inv_cnt : 0.f);
        if (use_l && u >= 0 && u < n) {
          // the mean through the hardware reciprocal (within an ulp or two
          // of the quotient; an IEEE division costs ten instructions a wave)
          const int lo = max(0, u - r), hi = min(n - 1, u + r);
          v += Vs[q] * __builtin_amdgcn_rcpf((float)(hi - lo + 1));
        }
        // B and V are 0 outside the candidates: the pool windows need no
        // per-position bounds either
        const bool cand = u >= 0 && u < nc;
        Bs[q] = cand ? bv[j] : 0.f;
        Vs[q] = cand ? v : 0.f;
      }
    }
    if (t < TAPS) {
      Bs[kSegWin + t] = 0.f;
      Vs[kSegWin + t] = 0.f;
    }
  }
  lds_barrier();

  // V, and the pooled B and V over I (truncated windows), of the segment's
  // candidates: two consecutive candidates per thread, whose 2hp + 1 taps
  // overlap, each summed in position order (a tap outside the candidates
  // adds 0)
  const int hp = a.pool_half;
  const int ncand = max(0, min(i0 + kSegLen, nc) - i0);
  float xb[PER], xv[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int q = t + j * NT;
    xb[j] = Bs[kPoolHalo + q];
    xv[j] = Vs[kPoolHalo + q];
  }
  {
    static_assert(PER == 2, "two consecutive candidates per thread");
    const int q0 = 2 * t;
    const float *bp = Bs + kPoolHalo + q0 - hp, *vp = Vs + kPoolHalo + q0 - hp;   // tap k of q0 (k <= 2hp)
    float b0 = bp[0], v0 = vp[0], b1 = 0.f, v1 = 0.f;
#pragma unroll 4
    for (int k = 1; k <= 2 * hp; ++k) {
      const float x = bp[k], y = vp[k];
      b0 += x; b1 += x; v0 += y; v1 += y;
    }
    b1 += bp[2 * hp + 1];
    v1 += vp[2 * hp + 1];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int q = q0 + j, i = i0 + q;
      if (q < ncand) {
        const float inv = __builtin_amdgcn_rcpf((float)(min(nc - 1, i + hp) - max(0, i - hp) + 1));
        a.vec_pB[base + i] = (j ? b1 : b0) * inv;
        a.vec_pV[base + i] = (j ? v1 : v0) * inv;
        a.vec_V[base + i] = Vs[kPoolHalo + q];
      }
    }
  }
  if (!calib) return;

  // boundary bin of the top-M of B, and the segment's list of candidates at
  // or above it (key, position, V) in position order
  unsigned cb[kHPer];
#pragma unroll
  for (int q = 0; q < kHPer / 4; ++q) {
    u32x4 x = hv[0][q];
#pragma unroll
    for (int c = 1; c < kHCopies; ++c) x += hv[c][q];
    cb[4 * q + 0] = x.x; cb[4 * q + 1] = x.y; cb[4 * q + 2] = x.z; cb[4 * q + 3] = x.w;
  }
  bins_boundary<kHPer, NT>(cb, M, ss);
  const int beta = ss.bc_i[0], above = ss.bc_i[1];
  const unsigned cntb = ss.bc_u[2];
  uint32_t msk = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j)
    msk |= (t + j * NT < ncand && hbin(float_key(xb[j])) >= beta ? 1u : 0u) << j;
  ordered_bases<PER, NT>(msk, pre);
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const bool in = (msk >> j) & 1u;
    const uint64_t m = __ballot(in);
    if (in) {
      const int64_t o = base + i0 + pre[j * NW + wave] + lane_rank(m);
      a.listB_key[o] = float_key(xb[j]);
      a.listB_pos[o] = i0 + t + j * NT;
      a.listB_v[o] = xv[j];
    }
  }
  if (t == 0) a.cntB[(int64_t)h * st.total_segs + gs] = (int)pre[PER * NW];
  if (sg == 0 && t == 0) a.recB[b * a.Hkv + h] = make_int4(beta, above, M - above, (int)cntb);
}

__global__ __launch_bounds__(kSegThreads) void k_segcal(SegArgs a, SeqTable st) {
  segcal_body(a, st, blockIdx.x, blockIdx.y, find_seg(st, blockIdx.x));
}

// Loads the selection record and the segments' lists of a (sequence, KV
// head) into registers as one sequence of entries e = t + j*NT in (segment,
// slot) order, which is position order.  First round: kListSpec slots per
// thread, every slot a segment may hold up to cs = kListSpec*NT/nseg (a
// multiple of 64; none beyond 32 segments), loaded with the counts in flight
// alongside.  When a count exceeds cs, a second round loads the exact entries
// from the counts' prefix (up to kListCap).  Entries that do not exist get
// key 0.  `fits` is false when the lists exceed kListCap.  scnt is LDS for
// kMaxSegs values.  Ends with a barrier.
template <bool WITH_V>
__device__ __forceinline__ void load_lists(const SeqTable &st, int b, int64_t base, int n, int h,
                                           const int4 *recp, const unsigned *lkey, const int *lpos,
                                           const float *lv, const int *cnts, int *scnt, ListView &L,
                                           int4 &rec, unsigned *k, int *p, float *v) {
  constexpr int NT = kSegThreads;
  const int t = threadIdx.x;
  L.nseg = st.seg_base[b + 1] - st.seg_base[b];
  const int cs = ((kListSpec * NT / L.nseg) / 64) * 64;
  L.cap = cs;
  const int tt = opaque(t);
  rec = *recp;                                   // first: it heads the longest chain
  // unconditional (clamped) so that no branch waits for the loads in flight
  int c = cnts[(int64_t)h * st.total_segs + st.seg_base[b] + min(tt, L.nseg - 1)];
  const int csd = max(cs, 64);    // the addressing only (no first round when cs is 0)
#pragma unroll
  for (int j = 0; j < kListSpec; ++j) {
    const int e = tt + j * NT, s = min(e / csd, L.nseg - 1);
    const int64_t o = base + min(s * kSegLen + (e - s * csd), n - 1);
    k[j] = lkey[o];
    p[j] = lpos[o];
    if constexpr (WITH_V) v[j] = lv[o];
  }
  // the record is uniform: taken here, so that moving it to scalar registers
  // waits for it only after the list loads are issued
  asm volatile("" : "+v"(rec.x), "+v"(rec.y), "+v"(rec.z), "+v"(rec.w));
#pragma unroll
  for (int j = kListSpec; j < kListPer; ++j) k[j] = 0u;
  if (t < kMaxSegs) scnt[t] = t < L.nseg ? c : 0;
  lds_barrier();
  // every thread reads all counts: no second barrier, no wait for the lists
  bool over = cs == 0;
  for (int s = 0; s < L.nseg; ++s) over |= scnt[s] > cs;
  if (!over) {
    L.fits = true;
#pragma unroll
    for (int j = 0; j < kListSpec; ++j) {
      const int e = t + j * NT, s = e / cs;
      if (s >= L.nseg || e - s * cs >= scnt[s]) k[j] = 0u;   // 0: not an entry
    }
    return;
  }
  // second round: exact entries after the counts' prefix (inclusive, in
  // place), each entry's segment found by bisection
  lds_barrier();
  if (t < 64) {
    const unsigned c0 = t < kMaxSegs ? (unsigned)scnt[t] : 0u;
    const unsigned inc = wave_incl_sum_u(c0);
    if (t < kMaxSegs) scnt[t] = (int)inc;
  }
  lds_barrier();
  const int total = scnt[L.nseg - 1];
  L.fits = total <= kListCap;
  if (!L.fits) return;
#pragma unroll
  for (int j = 0; j < kListPer; ++j) {
    const int e = t + j * NT;
    int lo = 0, hi = L.nseg - 1;          // the first segment whose prefix exceeds e
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (scnt[mid] > e) hi = mid; else lo = mid + 1;
    }
    const int before = lo > 0 ? scnt[lo - 1] : 0;
    const int64_t o = base + min(lo * kSegLen + (e - before), n - 1);
    k[j] = e < total ? lkey[o] : 0u;
    p[j] = lpos[o];
    if constexpr (WITH_V) v[j] = lv[o];
  }
}

// whole_moments beyond the register form (nc > kAllPer * NT): the threshold
// from global memory, then the members' moments in one more pass.
__device__ __forceinline__ void whole_moments_stream(const SegArgs &a, int64_t base, int nc,
                                                                int M, const unsigned *gh,
                                                                SelSharedT<kSegThreads> &ss,
                                                                double *part) {
  constexpr int NT = kSegThreads;
  const int t = threadIdx.x;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  unsigned xm;
  int pm;
  stream_threshold<kHCopies>(gh, [&](int i) { return float_key(a.vec_B[base + i]); }, nc, M, xm, pm, ss);
  const double bref = (double)key_float(xm), vref = (double)a.vec_V[base + pm];
  for (int i = t; i < nc; i += NT) {
    const float bv = a.vec_B[base + i];
    const unsigned x = float_key(bv);
    if (x > xm || (x == xm && i <= pm)) {
      const double db = (double)bv - bref, dv = (double)a.vec_V[base + i] - vref;
      s0 += db; s1 += db * db; s2 += dv; s3 += dv * dv;
    }
  }
  part[0] = s0; part[1] = s1; part[2] = s2; part[3] = s3; part[4] = bref;
}

// whole_topk beyond the register form: the threshold from global memory,
// then the members in position order over contiguous ranges of positions.
__device__ __forceinline__ void whole_topk_stream(const SegArgs &a, int64_t base, int nc,
                                                             int kept, const unsigned *gh, int32_t *idx,
                                                             int *tbl, SelSharedT<kSegThreads> &ss) {
  constexpr int NT = kSegThreads;
  const int t = threadIdx.x;
  unsigned xk;
  int pk;
  stream_threshold<1>(gh, [&](int i) { return a.vec_S[base + i]; }, nc, kept, xk, pk, ss);
  const int ch = (nc + NT - 1) / NT;
  const int i0 = min(nc, t * ch), i1 = min(nc, i0 + ch);
  auto member = [&](int i) {
    const unsigned x = a.vec_S[base + i];
    return x != 0u && (x > xk || (x == xk && i <= pk));
  };
  unsigned c = 0;
  for (int i = i0; i < i1; ++i) c += member(i) ? 1u : 0u;
  unsigned o = block_excl_scan_u<NT>(c, ss);
  for (int i = i0; i < i1; ++i)
    if (member(i)) {
      if (o < (unsigned)kept) {
        if (idx) idx[o] = i;
        tbl[o] = i;
      }
      ++o;
    }
}

// Scale-matching set and the thread's part of its moments over every
// candidate of a sequence, for lists beyond one workgroup: the B of all
// candidates in registers, the exact threshold over them; V is read for the
// members only.  Kept out of line so that its registers do not weigh on the
// list path of the calling kernel.
__device__ __attribute__((noinline)) void whole_moments(const SegArgs &a, int64_t base, int nc, int M,
                                                         const unsigned *gh, SelSharedT<kSegThreads> &ss,
                                                         unsigned *ckey, int *cpos, unsigned *pre,
                                                         float2 *mom, double *part) {
  constexpr int NT = kSegThreads, NW = NT / 64;
  const int t = threadIdx.x, wave = t >> 6;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
  float xb[kAllPer];
  {
    const int tt = opaque(t);
#pragma unroll
    for (int j = 0; j < kAllPer; ++j) xb[j] = a.vec_B[base + min(tt + j * NT, nc - 1)];
  }
  auto keyB = [&](int j) -> unsigned { return t + j * NT < nc ? float_key(xb[j]) : 0u; };
  auto posf = [&](int j) -> int { return t + j * NT; };
  unsigned xm;
  int pm;
  hist_threshold<kAllPer, kHCopies>(gh, keyB, posf, M, xm, pm, ss, ckey, cpos);
  uint32_t msk = 0;
#pragma unroll
  for (int j = 0; j < kAllPer; ++j) {
    const unsigned kj = keyB(j);
    msk |= (kj != 0u && (kj > xm || (kj == xm && posf(j) <= pm)) ? 1u : 0u) << j;
  }
  ordered_bases<kAllPer, NT>(msk, pre);
  // both moments are taken from values shifted by the boundary member's
  const double bref = (double)key_float(xm), vref = (double)a.vec_V[base + pm];
  for (int r0 = 0; r0 < M; r0 += kMomChunk) {
#pragma unroll
    for (int j = 0; j < kAllPer; ++j) {
      const bool in = (msk >> j) & 1u;
      const uint64_t m = __ballot(in);
      if (in) {
        const int o = (int)(pre[j * NW + wave] + lane_rank(m)) - r0;
        if (o >= 0 && o < kMomChunk) mom[o] = make_float2(xb[j], a.vec_V[base + t + j * NT]);
      }
    }
    lds_barrier();
    const int cnt = min(kMomChunk, M - r0);
    for (int e = t; e < cnt; e += NT) {
      const double db = (double)mom[e].x - bref, dv = (double)mom[e].y - vref;
      s0 += db; s1 += db * db; s2 += dv; s3 += dv * dv;
    }
    lds_barrier();
  }
  part[0] = s0; part[1] = s1; part[2] = s2; part[3] = s3; part[4] = bref;
}

// Score kernel (segment_score).
// (The select bodies take their arguments by value: a reference to a kernel
// argument that reaches an out-of-line call costs a stack copy and spills.)
__device__ __forceinline__ void segscore_body(SegArgs a, const SeqTable &st, int gs, int h, int b) {
  constexpr int NT = kSegThreads, PER = kSegPer, NW = NT / 64;
  __shared__ unsigned hist[kHBins];
  __shared__ unsigned ckey[kSegCandCap];
  __shared__ int cpos[kSegCandCap];
  __shared__ SelSharedT<NT> ss;
  __shared__ unsigned pre[kAllPer * NW + 1];
  __shared__ __align__(16) float2 mom[kMomChunk];
  __shared__ __align__(16) int scnt[kMaxSegs];
  __shared__ float vref_s;
  const int t = threadIdx.x;
  const int wave = t >> 6;
  const int sg = gs - st.seg_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int i0 = sg * kSegLen;
  const int ncand = max(0, min(i0 + kSegLen, nc) - i0);
  const int64_t base = (int64_t)h * a.T + st.cu[b];
  const int64_t hrow = ((int64_t)b * a.Hkv + h) * kHBins;
  for (int q = t; q < kHBins; q += NT) hist[q] = 0u;

  // what the pooled score is made of does not depend on lambda: in flight
  // first.  Mean of S: the pooled B and V (pool(B + lambda V) = pool(B) +
  // lambda pool(V)); mean of B before calibration: pooled B and V itself.
  // (The max of S reads B and V over the widened segment after lambda.)
  const bool max_s = a.pool_mode == POOL_MAX_S;
  float pb[PER], pv[PER];
  {
    const float *vsrc = a.pool_mode == POOL_MEAN_B ? a.vec_V : a.vec_pV;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int q = min(t + j * NT, max(ncand - 1, 0));
      pb[j] = max_s ? 0.f : a.vec_pB[base + i0 + q];
      pv[j] = max_s ? 0.f : vsrc[base + i0 + q];
    }
  }

  int M = scale_set_size(a.rho, sel_head_budget(st, a.hb, a.Hkv, b, h, a.sb));
  M = max(0, min(M, nc));
  float lam = 0.f;
  if (M > 0 && a.use_last_query) {
    int4 rec;                                          // boundary bin, above, need, its count
    unsigned lk[kListPer];
    int lp[kListPer];
    float lv[kListPer];
    ListView L;
    load_lists<true>(st, b, base, n, h, a.recB + b * a.Hkv + h, a.listB_key, a.listB_pos, a.listB_v,
                     a.cntB, scnt, L, rec, lk, lp, lv);
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0, bref_set = 0.0;
    if (L.fits && rec.w <= kSegCandCap) {
      // the boundary bin's entries, ranked under the tie rule
      compact_ballot<kListPer, NT, kSegCandCap>([&](int j) { return lk[j] != 0u && hbin(lk[j]) == rec.x; },
                                   [&](int j) { return lk[j]; }, [&](int j) { return lp[j]; },
                                   ckey, cpos, ss);
      unsigned xm;
      int pm;
      rank_pick_bin<NT>(rec.w, rec.z, ckey, cpos, ss, xm, pm);
      // population moments over the set in double, from values shifted by
      // the boundary member's (its B is the set's smallest; the thread that
      // holds the member posts its V): equal values give exactly 0
#pragma unroll
      for (int j = 0; j < kListPer; ++j)
        if (lk[j] == xm && lp[j] == pm) vref_s = lv[j];
      lds_barrier();
      const double bref = (double)key_float(xm), vref = (double)vref_s;
      bref_set = bref;
#pragma unroll
      for (int j = 0; j < kListPer; ++j) {
        if (lk[j] != 0u && (lk[j] > xm || (lk[j] == xm && lp[j] <= pm))) {
          const double db = (double)key_float(lk[j]) - bref, dv = (double)lv[j] - vref;
          s0 += db; s1 += db * db; s2 += dv; s3 += dv * dv;
        }
      }
    } else {
      double part[5];
      if (nc > kAllPer * kSegThreads)
        whole_moments_stream(a, base, nc, M, a.hist_B + hrow * kHCopies, ss, part);
      else
        whole_moments(a, base, nc, M, a.hist_B + hrow * kHCopies, ss, ckey, cpos, pre, mom, part);
      s0 = part[0]; s1 = part[1]; s2 = part[2]; s3 = part[3];
      bref_set = part[4];
    }
    // the moment scratch is free here (its fallback user is done)
    lam = block_lambda<NT>(s0, s1, s2, s3, M, bref_set, a.gamma, a.eps, a.b_floor,
                           reinterpret_cast<double *>(mom), ss, &vref_s);
  }
  if (sg == 0 && t == 0) {
    a.lambda_ws[b * a.Hkv + h] = lam;
    if (a.out_lambda) a.out_lambda[b * a.Hkv + h] = lam;
  }

  // pooled score keys of the segment, and their histogram
  lds_barrier();
  if (max_s) {
    // S over the segment widened by the pool halo in LDS (the moment scratch
    // is free now), -inf outside the candidate set, then the max over each
    // pool window
    float *sw = reinterpret_cast<float *>(mom);
    const int w0 = i0 - kPoolHalo;                   // position of window slot 0
    float wb[kSegWinJ], wv[kSegWinJ];
#pragma unroll
    for (int j = 0; j < kSegWinJ; ++j) {
      const int u = min(max(w0 + t + j * NT, 0), n - 1);
      wb[j] = a.vec_B[base + u];
      wv[j] = a.vec_V[base + u];
    }
#pragma unroll
    for (int j = 0; j < kSegWinJ; ++j) {
      const int q = t + j * NT, u = w0 + q;
      if (q < kSegWin) sw[q] = (u >= 0 && u < nc) ? fmaf(lam, wv[j], wb[j]) : -INFINITY;
    }
    lds_barrier();
    const int hp = a.pool_half;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int q = t + j * NT;
      if (q < ncand) {
        const int i = i0 + q, lo = max(0, i - hp), hi = min(nc - 1, i + hp);
        float mx = sw[lo - w0];
        for (int u = lo + 1; u <= hi; ++u) mx = fmaxf(mx, sw[u - w0]);
        const unsigned key = float_key(mx);
        a.vec_S[base + i] = key;
        atomicAdd(&hist[hbin(key)], 1u);
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int q = t + j * NT;
      if (q < ncand) {
        const unsigned key = float_key(fmaf(lam, pv[j], pb[j]));
        a.vec_S[base + i0 + q] = key;
        atomicAdd(&hist[hbin(key)], 1u);
      }
    }
  }
  lds_barrier();
  unsigned *gh = a.hist_S + hrow;
  for (int q = t; q < kHBins; q += NT) {
    const unsigned c = hist[q];
    if (c) atomicAdd(&gh[q], c);
  }
}

// Candidate kernel (segment_cand): the boundary bin of the top-K of the
// pooled score and the segment's list of entries at or above it.
__device__ __forceinline__ void segcand_body(SegArgs a, const SeqTable &st, int gs, int h, int b) {
  constexpr int NT = kSegThreads, PER = kSegPer, NW = NT / 64;
  __shared__ SelSharedT<NT> ss;
  __shared__ unsigned pre[PER * NW + 1];
  const int t = threadIdx.x;
  const int wave = t >> 6;
  const int sg = gs - st.seg_base[b];
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int i0 = sg * kSegLen;
  const int ncand = max(0, min(i0 + kSegLen, nc) - i0);
  const int64_t base = (int64_t)h * a.T + st.cu[b];
  const int kept = min(sel_head_budget(st, a.hb, a.Hkv, b, h, a.sb), nc);
  if (kept <= 0 || kept == nc) return;               // none or all kept: no list needed
  unsigned cb[kHPer];
  load_bins<1>(a.hist_S + ((int64_t)b * a.Hkv + h) * kHBins, cb);
  unsigned key[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) key[j] = a.vec_S[base + i0 + min(t + j * NT, max(ncand - 1, 0))];
  bins_boundary<kHPer, NT>(cb, kept, ss);
  const int beta = ss.bc_i[0], above = ss.bc_i[1];
  const unsigned cntb = ss.bc_u[2];
  uint32_t msk = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) msk |= (t + j * NT < ncand && hbin(key[j]) >= beta ? 1u : 0u) << j;
  ordered_bases<PER, NT>(msk, pre);
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const bool in = (msk >> j) & 1u;
    const uint64_t m = __ballot(in);
    if (in) {
      const int64_t o = base + i0 + pre[j * NW + wave] + lane_rank(m);
      a.listS_key[o] = key[j];
      a.listS_pos[o] = i0 + t + j * NT;
    }
  }
  if (t == 0) a.cntS[(int64_t)h * st.total_segs + gs] = (int)pre[PER * NW];
  if (sg == 0 && t == 0) a.recS[b * a.Hkv + h] = make_int4(beta, above, kept - above, (int)cntb);
}

// Top-K over every candidate of a sequence for lists beyond one workgroup:
// the pooled score keys of all candidates in registers, the exact threshold
// over them, the kept positions in ascending order into tbl (and idx unless
// it is null).  Kept out of line like whole_moments.
__device__ __attribute__((noinline)) void whole_topk(const SegArgs &a, int64_t base, int nc, int kept,
                                                      const unsigned *gh, int32_t *idx, int *tbl,
                                                      SelSharedT<kSegThreads> &ss, unsigned *ckey,
                                                      int *cpos, unsigned *pre) {
  constexpr int NT = kSegThreads, NW = NT / 64;
  const int t = threadIdx.x, wave = t >> 6;
  unsigned key[kAllPer];
  {
    const int tt = opaque(t);
#pragma unroll
    for (int j = 0; j < kAllPer; ++j) key[j] = a.vec_S[base + min(tt + j * NT, nc - 1)];
#pragma unroll
    for (int j = 0; j < kAllPer; ++j) if (tt + j * NT >= nc) key[j] = 0u;
  }
  auto keyS = [&](int j) -> unsigned { return key[j]; };
  auto posf = [&](int j) -> int { return t + j * NT; };
  unsigned xk;
  int pk;
  hist_threshold<kAllPer, 1>(gh, keyS, posf, kept, xk, pk,
                          ss, ckey, cpos);
  uint32_t msk = 0;
#pragma unroll
  for (int j = 0; j < kAllPer; ++j)
    msk |= (key[j] != 0u && (key[j] > xk || (key[j] == xk && posf(j) <= pk)) ? 1u : 0u) << j;
  // element j of thread t is position t + j*NT, so slot order is position order
  ordered_bases<kAllPer, NT>(msk, pre);
#pragma unroll
  for (int j = 0; j < kAllPer; ++j) {
    const bool in = (msk >> j) & 1u;
    const uint64_t m = __ballot(in);
    if (in) {
      const unsigned o = pre[j * NW + wave] + lane_rank(m);
      if (o < (unsigned)kept) {
        if (idx) idx[o] = posf(j);
        tbl[o] = posf(j);
      }
    }
  }
}

// Final kernel (final_topk): `parts` workgroups per (sequence, KV head)
// select the same top-K; part 0 writes the indices, each part gathers its
// share of the compacted rows (kept positions, the W window rows, zero rows
// up to K + W).
__device__ __forceinline__ void final_body(SegArgs a, const SeqTable &st, int part, int b,
                                           int h) {
  constexpr int NT = kSegThreads, NW = NT / 64;
  extern __shared__ __align__(16) int tbl[];         // [K + W] source position of each row
  __shared__ unsigned ckey[kSegCandCap];
  __shared__ int cpos[kSegCandCap];
  __shared__ SelSharedT<NT> ss;
  __shared__ unsigned pre[kAllPer * NW + 1];
  __shared__ __align__(16) int scnt[kMaxSegs];
  const int t = threadIdx.x;
  const int wave = t >> 6;
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int K = sel_head_budget(st, a.hb, a.Hkv, b, h, a.sb);   // this head's budget
  const int C = a.flat_heads ? K : sel_seq_budget(st, a.sb, b);  // rows of the head's block, less W
  const int kept = min(K, nc);
  const int64_t base = (int64_t)h * a.T + st.cu[b];
  int32_t *idx = a.idx + sel_head_idx_base(st, a.hb, a.Hkv, b, h, a.sb);
  if (kept > 0 && kept == nc) {
    // every candidate is kept
    for (int j = t; j < nc; j += NT) {
      if (part == 0) idx[j] = j;
      tbl[j] = j;
    }
  } else if (kept > 0) {
    // rows no member fills stay empty: the selection below sets exactly
    // `kept` of them, and this keeps a table row from ever holding a stale
    // position (the barriers of the list loads order it before those writes)
    for (int j = t; j < kept; j += NT) tbl[j] = -1;
    int4 rec;
    unsigned lk[kListPer];
    int lp[kListPer];
    ListView L;
    load_lists<false>(st, b, base, n, h, a.recS + b * a.Hkv + h, a.listS_key, a.listS_pos, nullptr,
                      a.cntS, scnt, L, rec, lk, lp, nullptr);
    if (L.fits && rec.w <= kSegCandCap) {
      compact_ballot<kListPer, NT, kSegCandCap>([&](int j) { return lk[j] != 0u && hbin(lk[j]) == rec.x; },
                                   [&](int j) { return lk[j]; }, [&](int j) { return lp[j]; },
                                   ckey, cpos, ss);
      unsigned xk;
      int pk;
      rank_pick_bin<NT>(rec.w, rec.z, ckey, cpos, ss, xk, pk);
      uint32_t msk = 0;
#pragma unroll
      for (int j = 0; j < kListPer; ++j)
        msk |= (lk[j] != 0u && (lk[j] > xk || (lk[j] == xk && lp[j] <= pk)) ? 1u : 0u) << j;
      // entries are in (segment, slot) = position order
      ordered_bases<kListPer, NT>(msk, pre);
#pragma unroll
      for (int j = 0; j < kListPer; ++j) {
        const bool in = (msk >> j) & 1u;
        const uint64_t m = __ballot(in);
        if (in) {
          const unsigned o = pre[j * NW + wave] + lane_rank(m);
          if (o < (unsigned)kept) {              // exactly `kept` are set; the bound guards the buffers
            if (part == 0) idx[o] = lp[j];
            tbl[o] = lp[j];
          }
        }
      }
    } else {
      if (nc > kAllPer * kSegThreads)
        whole_topk_stream(a, base, nc, kept, a.hist_S + ((int64_t)b * a.Hkv + h) * kHBins,
                          part == 0 ? idx : nullptr, tbl, ss);
      else
        whole_topk(a, base, nc, kept, a.hist_S + ((int64_t)b * a.Hkv + h) * kHBins, part == 0 ? idx : nullptr,
                 tbl, ss, ckey, cpos, pre);
    }
  }
  if (part == 0)
    for (int j = max(kept, 0) + t; j < K; j += NT) idx[j] = -1;
  for (int w = t; w < a.W; w += NT) tbl[kept + w] = nc + w;
  for (int j = kept + a.W + t; j < C + a.W; j += NT) tbl[j] = -1;
  lds_barrier();

  {
    // clear this part's slice of the B histogram for the next layer (its
    // readers, the calibration and score kernels, are done)
    constexpr int HB = kHCopies * kHBins;
    const int sl = 4 * ((HB / 4 + a.parts - 1) / a.parts);
    unsigned *hb = a.hist_B + ((int64_t)b * a.Hkv + h) * HB;
    for (int q = part * sl + 4 * t; q < min(HB, (part + 1) * sl); q += 4 * NT)
      *reinterpret_cast<u32x4 *>(hb + q) = u32x4{0u, 0u, 0u, 0u};
  }

  // this part's rows of the compacted cache
  const int rows = C + a.W;
  const int per = (rows + a.parts - 1) / a.parts;
  const int r0 = part * per, r1 = min(rows, r0 + per);
  const int pieces = a.row_bytes / 16;
  const int total = max(0, r1 - r0) * pieces;
  const unsigned char *ks = static_cast<const unsigned char *>(a.k);
  const unsigned char *vs = static_cast<const unsigned char *>(a.v);
  unsigned char *ko = static_cast<unsigned char *>(a.k_out);
  unsigned char *vo = static_cast<unsigned char *>(a.v_out);
  const int kept_base = sel_seq_kept_base(st, a.sb, b);
  constexpr int BATCH = 4;
  for (int q0 = t; q0 < total; q0 += BATCH * NT) {
    u32x4 kv[BATCH], vv[BATCH];
    int srcs[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int q = min(q0 + u * NT, total - 1);
      const int rr = r0 + q / pieces, p = q % pieces;
      const int src = tbl[rr];
      srcs[u] = (src >= 0 && src < n) ? src : -1;   // anything else is an empty row
      const int64_t so = ((int64_t)(st.cu[b] + max(srcs[u], 0)) * a.Hkv + h) * a.row_bytes + 16 * p;
      kv[u] = *reinterpret_cast<const u32x4 *>(ks + so);
      vv[u] = *reinterpret_cast<const u32x4 *>(vs + so);
    }
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int q = q0 + u * NT;
      if (q < total) {
        const int rr = r0 + q / pieces, p = q % pieces;
        const int64_t row = a.flat_heads
            ? (int64_t)a.Hkv * kept_base + a.hb[b * a.Hkv + h].y + (int64_t)h * a.W + rr
            : (int64_t)(kept_base + rr) * a.Hkv + h;
        const int64_t dst = row * a.row_bytes + 16 * p;
        const u32x4 z = u32x4{0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4 *>(ko + dst) = srcs[u] >= 0 ? kv[u] : z;
        *reinterpret_cast<u32x4 *>(vo + dst) = srcs[u] >= 0 ? vv[u] : z;
      }
    }
  }
}

__global__ __launch_bounds__(kSegThreads) void k_segscore(SegArgs a, SeqTable st) {
  segscore_body(a, st, blockIdx.x, blockIdx.y, find_seg(st, blockIdx.x));
}

__global__ __launch_bounds__(kSegThreads) void k_segcand(SegArgs a, SeqTable st) {
  segcand_body(a, st, blockIdx.x, blockIdx.y, find_seg(st, blockIdx.x));
}

__global__ __launch_bounds__(kSegThreads) void k_segfinal(SegArgs a, SeqTable st) {
  final_body(a, st, blockIdx.x, blockIdx.y, blockIdx.z);
}

// Launches that carry work of two or three layers (a prompt's layers in
// flight at once; the jobs of one launch share no buffer, see the host's
// schedule):
//  * k_sel_a, jobs along blockIdx.y and KV heads along blockIdx.x: [0, nseg)
//    the calibration of this layer (g), [nseg, nseg + ncand) the candidate
//    lists of the previous layer (gp), then the next layer's row
//    normalisers (m; each workgroup takes kSegThreads / kMergeThreads row
//    groups of a sequence).  Workgroups are dispatched x first, so every
//    head's calibration (the longest job) is dispatched before any shorter
//    one, and a grid beyond one round of the CUs leaves short jobs waiting.
//  * k_sel_b, jobs along blockIdx.x per KV head (blockIdx.y): [0, nfinal)
//    the final top-K and compaction of the previous layer (parts per
//    sequence), then the scores of this layer.
__global__ __launch_bounds__(kSegThreads) void k_sel_a(SegArgs g, SegArgs gp, PassArgs m, SeqTable st,
                                                      int ncand, int nmerge) {
  const int h = blockIdx.x, job = blockIdx.y, nseg = st.total_segs;
  if (job < nseg) {
    segcal_body(g, st, job, h, find_seg(st, job));
    return;
  }
  const int x = job - nseg;
  if (x < ncand) {
    segcand_body(gp, st, x, h, find_seg(st, x));
  } else if (x < ncand + nmerge) {
    constexpr int groups = kSegThreads / kMergeThreads;
    __shared__ float2 mrg[groups][kMergeParts][kMergeRows];
    const int per_seq = (m.Rpad / kMergeRows + groups - 1) / groups;
    const int q = x - ncand, b = q / per_seq;
    const int grp = threadIdx.x / kMergeThreads;
    const int rg = (q - b * per_seq) * groups + grp;
    merge_rows(m, st, rg, b, h, threadIdx.x % kMergeThreads, mrg[grp], rg * kMergeRows < m.Rpad);
  }
}

__global__ __launch_bounds__(kSegThreads) void k_sel_b(SegArgs g, SegArgs gp, SeqTable st, int nfinal) {
  const int h = blockIdx.y, nseg = st.total_segs, batch = st.batch;
  // both table words in one round of scalar loads (the job split below
  // would otherwise wait for each in turn); a batch of one sequence takes a
  // copy of the score body with b = 0, whose per-sequence table reads sit at
  // fixed kernel-argument offsets and need no sequence search first.  (Not
  // in k_sel_a: there the copies' scalar registers would cost the second
  // workgroup per CU, and they did not pay.)
  asm volatile("" ::"s"(nseg), "s"(batch));
  if ((int)blockIdx.x < nseg) {
    if (batch == 1)
      segscore_body(g, st, blockIdx.x, h, 0);
    else
      segscore_body(g, st, blockIdx.x, h, find_seg(st, blockIdx.x));
  } else {
    const int x = blockIdx.x - nseg;
    final_body(gp, st, x % gp.parts, x / gp.parts, h);
  }
  (void)nfinal;
}

size_t final_lds_bytes(int max_budget, int window) {
  return (size_t)(max_budget + window) * sizeof(int) + 2 * kSegCandCap * sizeof(unsigned) +
         sizeof(SelSharedT<kSegThreads>) + (kAllPer * (kSegThreads / 64) + 1) * sizeof(unsigned) +
         kMaxSegs * sizeof(int);
}

hipError_t launch_segcal(const SegArgs &a, const SeqTable &st, hipStream_t s) {
  dim3 grid(st.total_segs, a.Hkv), block(kSegThreads);
  hipLaunchKernelGGL(k_segcal, grid, block, 0, s, a, st);
  return hipGetLastError();
}

hipError_t launch_sel_a(const SegArgs &g, const SegArgs *gp, const PassArgs *m, const SeqTable &st,
                       hipStream_t s) {
  constexpr int groups = kSegThreads / kMergeThreads;
  int nmerge = 0;
  if (m) {
    if (m->Rpad % kMergeRows || m->Hkv != g.Hkv) return hipErrorInvalidValue;
    nmerge = st.batch * ((m->Rpad / kMergeRows + groups - 1) / groups);
  }
  const int ncand = gp ? st.total_segs : 0;
  dim3 grid(g.Hkv, ncand + nmerge + st.total_segs), block(kSegThreads);
  hipLaunchKernelGGL(k_sel_a, grid, block, 0, s, g, gp ? *gp : g, m ? *m : PassArgs{}, st, ncand,
                     nmerge);
  return hipGetLastError();
}

size_t sel_b_lds_bytes(int max_budget, int window) {
  hipFuncAttributes fa{};
  if (hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(k_sel_b)) != hipSuccess) return SIZE_MAX;
  return fa.sharedSizeBytes + (size_t)(max_budget + window) * sizeof(int);
}

hipError_t launch_sel_b(const SegArgs &g, const SegArgs *gp, const SeqTable &st, int max_budget,
                        hipStream_t s) {
  const size_t lds = gp ? (size_t)(max_budget + g.W) * sizeof(int) : 0;
  if (gp && (sel_b_lds_bytes(max_budget, g.W) > (size_t)kLdsBytes || gp->parts < 1))
    return hipErrorInvalidValue;
  const int nfinal = gp ? gp->parts * st.batch : 0;
  allow_lds(k_sel_b, lds);
  hipLaunchKernelGGL(k_sel_b, dim3(nfinal + st.total_segs, g.Hkv), dim3(kSegThreads), lds, s, g,
                     gp ? *gp : g, st, nfinal);
  return hipGetLastError();
}

hipError_t launch_segscore(const SegArgs &a, const SeqTable &st, hipStream_t s) {
  dim3 grid(st.total_segs, a.Hkv), block(kSegThreads);
  hipLaunchKernelGGL(k_segscore, grid, block, 0, s, a, st);
  return hipGetLastError();
}

hipError_t launch_segcand(const SegArgs &a, const SeqTable &st, hipStream_t s) {
  dim3 grid(st.total_segs, a.Hkv), block(kSegThreads);
  hipLaunchKernelGGL(k_segcand, grid, block, 0, s, a, st);
  return hipGetLastError();
}

hipError_t launch_segfinal(const SegArgs &a, const SeqTable &st, int max_budget, hipStream_t s) {
  const size_t lds = (size_t)(max_budget + a.W) * sizeof(int);
  if (final_lds_bytes(max_budget, a.W) > (size_t)kLdsBytes || a.parts < 1) return hipErrorInvalidValue;
  allow_lds(k_segfinal, lds);
  hipLaunchKernelGGL(k_segfinal, dim3(a.parts, st.batch, a.Hkv), dim3(kSegThreads), lds, s, a, st);
  return hipGetLastError();
}

// ---------------------------------------------------------------- head-wise allocation
// AdaKV's budget allocation of one (layer, sequence) (App. B: the backbone's
// head-wise budgets, kept under BACON).  Every KV head keeps its top
// f = floor(alpha K) positions by the backbone score A, the mean pool of B
// over the candidates; the other H (K - f) slots go to the highest A over the
// union of every head's remaining positions (ties: score desc, head asc,
// position asc).  Counted without sorting: with g_h(x) the head's entries
// above key x, the union's slots above x number F(x) = sum_h max(0, g_h(x) - f),
// so a radix search over the key digits (per-head histograms in LDS) finds
// the boundary key tau with F(above tau) < H (K - f) <= F(tau); the tie at tau
// goes to the lower heads, and K_h = f + the head's share.  One workgroup per
// sequence; A is written to a [Hkv, T] buffer between the passes.
constexpr int kAllocThreads = 1024;
constexpr int kAllocDigits = 1024;       // bins of a radix level (10 bits)
constexpr int kAllocTile = 4096;         // positions of B staged per round of the pool
constexpr int kMaxAllocHeads = 32;

size_t alloc_lds_bytes(int hkv) { return (size_t)hkv * kAllocDigits * sizeof(unsigned); }

__global__ __launch_bounds__(kAllocThreads) void k_alloc(AllocArgs a, SeqTable st) {
  constexpr int NT = kAllocThreads;
  extern __shared__ __align__(16) unsigned hist[];      // [Hkv][kAllocDigits]
  __shared__ float tile[kAllocTile + 2 * kPoolHalo];
  __shared__ SelSharedT<NT> ss;
  __shared__ unsigned above[kMaxAllocHeads], eq[kMaxAllocHeads];
  __shared__ int kh_s[kMaxAllocHeads];
  const int t = threadIdx.x, b = blockIdx.x, H = a.Hkv;
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int K = seq_budget(st, a.sb, b);
  int2 *tab = a.hb + (int64_t)b * H;
  if (nc <= K) {
    // every head keeps all its candidates: the budgets stay uniform
    for (int h = t; h < H; h += NT) {
      tab[h] = make_int2(K, h * K);
      if (a.out) a.out[(int64_t)b * H + h] = K;
    }
    return;
  }
  const int f = (int)min((double)K, floor(a.alpha * (double)K));
  const unsigned R = (unsigned)H * (unsigned)(K - f);
  const int ph = a.pool_half;
  const int64_t T = a.T, s0 = st.cu[b];

  // pass 0: A = the mean pool of B over the candidates (truncated at the
  // ends), written out, and the histograms of its top key digit
  for (int e = t; e < H * kAllocDigits; e += NT) hist[e] = 0u;
  for (int h = 0; h < H; ++h) {
    const float *B = a.vec_B + (int64_t)h * T + s0;
    float *A = a.vec_A + (int64_t)h * T + s0;
    for (int i0 = 0; i0 < nc; i0 += kAllocTile) {
      __syncthreads();
      const int lo = max(0, i0 - ph), hi = min(nc, i0 + kAllocTile + ph);
      for (int j = lo + t; j < hi; j += NT) tile[j - lo] = B[j];
      __syncthreads();
      for (int i = i0 + t; i < min(nc, i0 + kAllocTile); i += NT) {
        const int w0 = max(0, i - ph), w1 = min(nc - 1, i + ph);
        float acc = 0.f;
        for (int j = w0; j <= w1; ++j) acc += tile[j - lo];
        const float v = acc / (float)(w1 - w0 + 1);
        A[i] = v;
        atomicAdd(&hist[h * kAllocDigits + (float_key(v) >> 22)], 1u);
      }
    }
  }
  for (int h = t; h < H; h += NT) above[h] = 0u;
  __syncthreads();

  // radix levels over key bits 31..22, 21..12, 11..2, 1..0
  unsigned prefix = 0u;
  for (int lev = 0; lev < 4; ++lev) {
    const int shift = lev == 3 ? 0 : 22 - 10 * lev;
    const int width = lev == 3 ? 2 : 10;
    if (lev > 0) {
      for (int e = t; e < H * kAllocDigits; e += NT) hist[e] = 0u;
      __syncthreads();
      const int pshift = shift + width;
      for (int h = 0; h < H; ++h) {
        const float *A = a.vec_A + (int64_t)h * T + s0;
        for (int i = t; i < nc; i += NT) {
          const unsigned k = float_key(A[i]);
          if ((k >> pshift) == prefix)
            atomicAdd(&hist[h * kAllocDigits + ((k >> shift) & ((1u << width) - 1u))], 1u);
        }
      }
      __syncthreads();
    }
    // suffix sums per head in place: hist[h][x] = entries of head h with
    // this level's digit >= x (under the prefix)
    for (int h = 0; h < H; ++h) {
      const unsigned v = hist[h * kAllocDigits + (kAllocDigits - 1 - t)];
      const unsigned inc = block_excl_scan_u<NT>(v, ss) + v;
      hist[h * kAllocDigits + (kAllocDigits - 1 - t)] = inc;
      __syncthreads();
    }
    // F(x) at this thread's digit; the boundary is the largest x with F >= R
    unsigned F = 0u;
    for (int h = 0; h < H; ++h) {
      const unsigned g = above[h] + hist[h * kAllocDigits + t];
      F += g > (unsigned)f ? g - (unsigned)f : 0u;
    }
    // (some digit always qualifies: F at digit 0 counts the union at or
    // below the previous boundary; the clamp only keeps indexes in range)
    const unsigned xb = max(block_reduce_u<1, NT>(F >= R ? (unsigned)t + 1u : 0u, ss), 1u) - 1u;
    // the entries above the boundary digit join `above`; the boundary digit's
    // own count is kept for the last level
    if (t < H) {
      const unsigned at = hist[t * kAllocDigits + xb];
      const unsigned up = xb + 1 < (unsigned)kAllocDigits ? hist[t * kAllocDigits + xb + 1] : 0u;
      eq[t] = at - up;
      above[t] += up;
    }
    prefix = (prefix << width) | xb;
    __syncthreads();
  }

  // the tie at tau: each head's entries equal to tau beyond its floor, taken
  // in head order until the union's slots are filled
  if (t == 0) {
    unsigned got = 0u;
    for (int h = 0; h < H; ++h) got += above[h] > (unsigned)f ? above[h] - (unsigned)f : 0u;
    unsigned need = got < R ? R - got : 0u;
    int off = 0;
    bool ok = true;
    for (int h = 0; h < H; ++h) {
      const unsigned g = above[h], ge = g + eq[h];
      const unsigned hi2 = ge > (unsigned)f ? ge - (unsigned)f : 0u;
      const unsigned lo2 = g > (unsigned)f ? g - (unsigned)f : 0u;
      const unsigned take = min(hi2 - lo2, need);
      need -= take;
      kh_s[h] = f + (int)(lo2 + take);
      ok = ok && kh_s[h] <= nc;
      off += kh_s[h];
    }
    // the budgets fill the sequence's H K slots exactly (its idx region and
    // compacted rows); anything else would be a fault of the search above,
    // reported on the error word with the budgets left uniform
    if (!ok || off != H * K) {
      for (int h = 0; h < H; ++h) kh_s[h] = K;
      if (a.err) __hip_atomic_store(a.err, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    off = 0;
    for (int h = 0; h < H; ++h) {
      tab[h] = make_int2(kh_s[h], off);
      off += kh_s[h];
    }
  }
  __syncthreads();
  if (a.out)
    for (int h = t; h < H; h += NT) a.out[(int64_t)b * H + h] = kh_s[h];
}

hipError_t launch_alloc(const AllocArgs &a, const SeqTable &st, hipStream_t s) {
  if (a.Hkv < 1 || a.Hkv > kMaxAllocHeads || !a.vec_B || !a.vec_A || !a.hb) return hipErrorInvalidValue;
  const size_t lds = alloc_lds_bytes(a.Hkv);
  allow_lds(k_alloc, lds);
  hipLaunchKernelGGL(k_alloc, dim3(st.batch), dim3(kAllocThreads), lds, s, a, st);
  return hipGetLastError();
}

// ---------------------------------------------------------------- split calibrate
// One position per thread: E from B and Q (Eq. boundary_residual), T from the
// history, the full L over the sequence-truncated neighbourhood, history update.
__global__ __launch_bounds__(256) void k_elem(ElemArgs a, SeqTable st) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int h = blockIdx.y;
  if (g >= a.T) return;
  int b = 0;
  while (b + 1 < st.batch && st.cu[b + 1] <= g) ++b;
  const int s0 = st.cu[b], n = st.cu[b + 1] - s0;
  const int i = (int)(g - s0);
  const int64_t row = (int64_t)h * a.T;
  const int64_t pos = row + g;
  auto resid = [&](int64_t p) {
    const float Bv = a.in_B[p], Qv = a.in_Q[p];
    return (Qv > Bv) ? (Qv - Bv) : 0.f;
  };
  const float E = resid(pos);
  // T: the previous ring_cnt layers, oldest first
  float ts = 0.f;
  for (int j = a.ring_cnt; j >= 1; --j)
    ts += a.ring[((a.ring_write - j + a.ring_slots) % a.ring_slots) * a.ring_stride + pos];
  const float Tv = a.ring_cnt ? ts / (float)a.ring_cnt : 0.f;
  // part of L with neighbours inside the position's chunk, as the fused pass
  // forms it (the select kernel adds the neighbours across chunk boundaries)
  float L = 0.f;
  if (a.terms & 2u) {
    const int k0 = (i / a.chunk) * a.chunk, k1 = min(n, k0 + a.chunk);
    const int lo = max(0, i - a.radius), hi = min(n - 1, i + a.radius);
    float s = 0.f;
    for (int u = max(lo, k0); u <= min(hi, k1 - 1); ++u) s += resid(row + s0 + u);
    L = s / (float)(hi - lo + 1);
  }
  a.ring[a.ring_write * a.ring_stride + pos] = E;
  a.vec_VP[pos] = ((a.terms & 1u) ? E : 0.f) + ((a.terms & 4u) ? Tv : 0.f) + L;
}

hipError_t launch_elem(const ElemArgs &a, const SeqTable &st, hipStream_t s) {
  dim3 grid((unsigned)((a.T + 255) / 256), a.Hkv), block(256);
  hipLaunchKernelGGL(k_elem, grid, block, 0, s, a, st);
  return hipGetLastError();
}

// ---------------------------------------------------------------- fill
// Zeroes n 32-bit words (16-byte aligned, n a multiple of 4).
__global__ __launch_bounds__(256) void k_zero(unsigned *p, int64_t n) {
  for (int64_t q = 4 * ((int64_t)blockIdx.x * 256 + threadIdx.x); q < n; q += 4 * (int64_t)gridDim.x * 256)
    *reinterpret_cast<u32x4 *>(p + q) = u32x4{0u, 0u, 0u, 0u};
}

hipError_t launch_zero(unsigned *p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (n % 4 || reinterpret_cast<uintptr_t>(p) % 16) return hipErrorInvalidValue;
  const int64_t blocks = std::min<int64_t>(1024, (n / 4 + 255) / 256);
  hipLaunchKernelGGL(k_zero, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------- compaction
// Rows of the compacted cache of a (sequence, KV head): the kept positions of
// idx, the W window rows, then zero rows up to K + W.  Each thread moves
// kCompactPer 16-byte pieces of K and V, all loads issued before the stores.
constexpr int kCompactPer = 2;

__global__ __launch_bounds__(256) void k_compact(CompactArgs a, SeqTable st) {
  const int b = blockIdx.x, h = blockIdx.y;
  const int n = st.cu[b + 1] - st.cu[b];
  const int nc = n - a.W;
  const int K = head_budget(st, a.hb, a.Hkv, b, h);
  const int kept = min(K, nc);
  const int32_t *idx = a.idx + head_idx_base(st, a.hb, a.Hkv, b, h);
  const int pieces = a.row_bytes / 16;
  const int total = (st.budget[b] + a.W) * pieces;   // rows per head of the sequence
  const int q0 = blockIdx.z * (256 * kCompactPer) + threadIdx.x;
  if (q0 >= total) return;
  const unsigned char *ks = static_cast<const unsigned char *>(a.k);
  const unsigned char *vs = static_cast<const unsigned char *>(a.v);
  unsigned char *ko = static_cast<unsigned char *>(a.k_out);
  unsigned char *vo = static_cast<unsigned char *>(a.v_out);
  int src[kCompactPer];
#pragma unroll
  for (int u = 0; u < kCompactPer; ++u) {
    const int q = min(q0 + 256 * u, total - 1);
    const int r = q / pieces;
    const int s = idx[min(r, max(kept - 1, 0))];
    src[u] = r < kept ? ((s >= 0 && s < n) ? s : -1) : (r < kept + a.W ? nc + (r - kept) : -1);
  }
  u32x4 kv[kCompactPer], vv[kCompactPer];
#pragma unroll
  for (int u = 0; u < kCompactPer; ++u) {
    const int q = min(q0 + 256 * u, total - 1);
    const int p = q - (q / pieces) * pieces;
    const int64_t so = ((int64_t)(st.cu[b] + max(src[u], 0)) * a.Hkv + h) * a.row_bytes + 16 * p;
    kv[u] = *reinterpret_cast<const u32x4 *>(ks + so);
    vv[u] = *reinterpret_cast<const u32x4 *>(vs + so);
  }
#pragma unroll
  for (int u = 0; u < kCompactPer; ++u) {
    const int q = q0 + 256 * u;
    if (q < total) {
      const int r = q / pieces, p = q - r * pieces;
      const int64_t dst = ((int64_t)(st.kept_base[b] + r) * a.Hkv + h) * a.row_bytes + 16 * p;
      const u32x4 z = u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4 *>(ko + dst) = src[u] >= 0 ? kv[u] : z;
      *reinterpret_cast<u32x4 *>(vo + dst) = src[u] >= 0 ? vv[u] : z;
    }
  }
}

__global__ __launch_bounds__(kHbChunk) void k_set_hb(HbChunk c, int2 *dst) {
  if ((int)threadIdx.x < c.n) dst[c.base + threadIdx.x] = c.v[threadIdx.x];
}

hipError_t launch_set_hb(const HbChunk &c, int2 *dst, hipStream_t s) {
  hipLaunchKernelGGL(k_set_hb, dim3(1), dim3(kHbChunk), 0, s, c, dst);
  return hipGetLastError();
}

hipError_t launch_compact(const CompactArgs &a, const SeqTable &st, hipStream_t s) {
  int kmax = 0;
  for (int b = 0; b < st.batch; ++b) kmax = max(kmax, st.budget[b]);
  const int64_t total = (int64_t)(kmax + a.W) * (a.row_bytes / 16);
  const int z = (int)((total + 256 * kCompactPer - 1) / (256 * kCompactPer));
  if (z <= 0) return hipSuccess;
  dim3 grid(st.batch, a.Hkv, z), block(256);
  hipLaunchKernelGGL(k_compact, grid, block, 0, s, a, st);
  return hipGetLastError();
}

}  // namespace bacon
