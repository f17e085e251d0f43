// Internal declarations shared by the gfx950 kernels and the host API.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bacon {

constexpr int kMaxBatch = 64;       // sequences per batch (kernel-argument table)
constexpr int kMaxSeqLen = 131072;  // positions per sequence (the segment select of the fused calls)
constexpr int kMaxSelLen = 32768;   // positions per sequence of the split calls' block select (in LDS)
constexpr int kMaxRows = 256;       // G*W window rows per KV head (8 row tiles of 32)
constexpr int kMaxRing = 16;        // persistence depth m
constexpr int kMaxChunk = 4096;     // keys per pass workgroup
constexpr int kSelThreads = 1024;
constexpr int kSelPer = kMaxSelLen / kSelThreads;   // positions per select thread
constexpr int kHistBins = 2048;     // 11-bit digits of the block select
constexpr int kSegLen = 2048;       // positions per segment of the histogram select
constexpr int kSegThreads = 1024;
constexpr int kPoolHalo = 16;       // largest pool half-width
constexpr int kHBins = 8192;        // bins of the select histograms (32 per octave of a float)
constexpr int kHCopies = 1;         // copies of the B histogram the fused pass spreads its atomics over
constexpr int kLdsBytes = 160 * 1024;   // LDS per CU (and per workgroup) on gfx950
constexpr int kEdgeEntries = 1024;      // positions next to chunk boundaries the select stages
constexpr int kKrWaves = 4;             // waves of a key-register pass workgroup
constexpr int kSyncStride = 64;          // words between groups' meeting counters (own 256-byte lines)
// Static device scratch of the allocation-free entry point (per GPU).
constexpr size_t kStaticScratchBytes = 4u << 20;

// Per-sequence layout, passed by value to every kernel.
struct SeqTable {
  int32_t batch;
  int32_t total_chunks;                 // key chunks per KV head over the batch
  int32_t total_segs;                   // select segments per KV head over the batch
  int32_t seg_base[kMaxBatch + 1];      // first select segment of each sequence
  int32_t cu[kMaxBatch + 1];            // token offsets
  int32_t chunk_base[kMaxBatch + 1];    // first chunk of each sequence
  int32_t budget[kMaxBatch];            // kept keys per KV head (the largest head budget
                                        // when the heads have their own)
  int32_t idx_base[kMaxBatch];          // idx entries before sequence b (all its heads)
  int32_t kept_base[kMaxBatch];         // sum of (budget + W) before b
};

enum PassMode { PASS_LSE = 0, PASS_SCORE = 1, PASS_FUSED = 2 };

// Arguments of the two K-streaming passes.
struct PassArgs {
  const void *q;        // [B*W, Hq, d]
  const void *k;        // [T, Hkv, d]
  int Hq, Hkv, G, W, R, Rpad;
  int chunk;            // keys per chunk (multiple of the stage size)
  int64_t T;            // row length of the [Hkv, T] vectors
  float c2;             // log2(e) / sqrt(d)
  float2 *partials;     // [Hkv, total_chunks, Rpad]  (max, sum) per chunk, log2 units
  float *lse2;          // [B, Hkv, Rpad] row normalisers, log2 units (merge kernel writes)
  float *lse_user;      // optional [B, Hq, W] natural-log normaliser (merge kernel writes)
  const float *lse_in;  // optional [B, Hq, W] natural-log normalisers given by the caller (pass 2 reads)
  unsigned *hist_B;     // [B, Hkv, kHCopies, kHBins] B histogram of the select (fused pass adds)
  // PASS_SCORE
  float *out_B, *out_Q; // [Hkv, T]
  // PASS_FUSED
  float *ring;          // [slots, Hkv, T] E history; slot l % slots holds layer l
  int64_t ring_stride;  // Hkv * T, floats between slots
  int ring_write;       // slot receiving this layer's E
  float *vec_B;         // [Hkv, T] window score
  float *vec_VP;        // [Hkv, T] unused by the fused pass (the calibration kernel forms V)
  int radius;
  uint32_t terms;
  // single-read pass: per group (sequence, KV head) an arrival and a done
  // counter at sync[kSyncStride * group + {0, 1}], the error word at
  // sync[kSyncStride * sync_groups], and the published row normalisers
  // (bitwise complement of the float; 0 = not yet) at bcast[group * Rpad + row]
  unsigned *sync;
  unsigned *bcast;
  int sync_groups;
};

enum SelMode { SEL_CALIB = 1, SEL_TOPK = 2 };
enum PoolMode { POOL_MEAN_S = 0, POOL_MAX_S = 1, POOL_MEAN_B = 2 };

struct SelArgs {
  int Hkv, W;
  int64_t T;
  int radius, pool_half, pool_mode;
  int vp_chunk;            // chunk size of the in-chunk L partial in vec_VP
  double rho;              // scale-matching expansion (double: M = floor(rho K) as the oracle forms it)
  float gamma, eps;
  int use_last_query;
  uint32_t terms;
  const float *vec_B;      // [Hkv, T]
  const float *vec_VP;     // [Hkv, T]
  const float *ring;       // [slots, Hkv, T] E history
  int64_t ring_stride;     // Hkv * T
  int ring_slot;           // slot of this layer's E
  const float *in_S;       // SEL_TOPK: user S [Hkv, T]
  float *out_S, *out_V, *out_E;  // SEL_CALIB optional outputs [Hkv, T]
  float *out_lambda;       // optional [B, Hkv]
  float *lambda_ws;        // [B, Hkv]
  int32_t *idx;            // SEL_TOPK output
  const int2 *hb;          // optional [B, Hkv] (budget, idx offset in the sequence)
};

// Histogram select of the fused pass (calibration, score and final kernels).
struct SegArgs {
  int Hkv, W;
  int64_t T;
  int radius, pool_half, pool_mode, vp_chunk;
  double rho;                    // scale-matching expansion
  float gamma, eps;
  // relative rounding bound of B (0 when B is exact to fp32): a set whose
  // Std(B) is at most b_floor times its mean B has no spread B resolves, and
  // takes Std(B) = 0
  float b_floor;
  int use_last_query;
  uint32_t terms;
  const float *vec_B, *vec_VP;   // [Hkv, T]
  const float *ring;             // [slots, Hkv, T] E history
  int64_t ring_stride;           // Hkv * T
  int ring_slots, ring_slot;     // slot count; slot of this layer's E
  int ring_cnt;                  // earlier layers averaged into T: slots ring_slot - cnt .. ring_slot - 1
  float *vec_V;                  // [Hkv, T] V = E + L + T over I
  float *vec_pB, *vec_pV;        // [Hkv, T] pooled B and V over I
  unsigned *vec_S;               // [Hkv, T] keys of the pooled score over I
  unsigned *hist_B, *hist_S;     // key histograms of B [B, Hkv, kHCopies, kHBins] (the bin count is
                                 // the sum of the copies) and of the pooled score [B, Hkv, kHBins];
                                 // the final kernel clears hist_B for the next layer, the
                                 // calibration kernel clears hist_S
  // per-segment lists at or above a boundary bin: segment s of a sequence
  // writes slots [s*kSegLen, ...) of the [Hkv, T] arrays, its count to cnt
  unsigned *listB_key, *listS_key;
  int *listB_pos, *listS_pos;
  float *listB_v;
  int *cntB, *cntS;              // [Hkv, total_segs]
  int4 *recB, *recS;             // [B, Hkv] boundary bin, count above, rank in it, its count
  float *lambda_ws, *out_lambda; // [B, Hkv]
  int32_t *idx;
  const void *k, *v;             // gather of the final kernel
  void *k_out, *v_out;
  int row_bytes;
  int parts;                     // final-kernel workgroups per (sequence, KV head)
  const int2 *hb;                // optional [B, Hkv] (budget, idx offset in the sequence)
  const int4 *sb;                // optional [B] (budget, idx base, kept-row base, 0) of this
                                 // layer's batch, when it differs from the SeqTable's (a
                                 // per-layer budget schedule: a launch holds two layers' jobs)
  // compacted cache one head per row: sequence b's rows start at Hkv times
  // its kept-row base, head h's block (K_h kept rows, then W window rows) at
  // its idx offset plus h W rows (the head-wise allocation, whose budgets
  // the host does not know)
  int flat_heads;
};

// Head-wise budget allocation of one layer (AdaKV's rule): K_{b,h} from the
// pooled window score of every KV head of a sequence.
struct AllocArgs {
  int Hkv, W, pool_half;
  int64_t T;
  double alpha;                  // floor fraction: every head keeps floor(alpha K) at least
  const float *vec_B;            // [Hkv, T]
  float *vec_A;                  // [Hkv, T] scratch: the pooled B
  int2 *hb;                      // out [B, Hkv] (K_{b,h}, idx offset in the sequence)
  int32_t *out;                  // optional out [B, Hkv] K_{b,h}
  const int4 *sb;                // optional per-layer sequence table (budget K_b in .x)
  unsigned *err;                 // optional error word (set to 2 if the search fails)
};

struct ElemArgs {           // split calibrate: E, T, L, ring update
  const float *in_B, *in_Q;
  float *ring;
  int64_t ring_stride;
  int ring_slots, ring_write, ring_cnt;
  float *vec_VP;
  int Hkv, radius, chunk;
  int64_t T;
  uint32_t terms;
};

struct CompactArgs {
  const int32_t *idx;
  const void *k, *v;
  void *k_out, *v_out;
  int Hkv, W, row_bytes;
  const int2 *hb;          // optional [B, Hkv] (budget, idx offset in the sequence)
};

// Size of the scale-matching set before the |I| cap (Sec. 4.4, Eq.
// scale_matching_size): floor(rho K) with the product formed in double.
__host__ __device__ inline int scale_set_size(double rho, int K) {
  const double m = floor(rho * (double)K);
  return m > 2147483647.0 ? 2147483647 : (int)m;
}

// Per-sequence budget fields of a layer's batch: from the table sb when
// given, else from the SeqTable.  seq_budget is the largest budget of the
// sequence's heads (its rows per head in the compacted cache, less W).
__host__ __device__ inline int seq_budget(const SeqTable &st, const int4 *sb, int b) {
  return sb ? sb[b].x : st.budget[b];
}
__host__ __device__ inline int seq_idx_base(const SeqTable &st, const int4 *sb, int b) {
  return sb ? sb[b].y : st.idx_base[b];
}
__host__ __device__ inline int seq_kept_base(const SeqTable &st, const int4 *sb, int b) {
  return sb ? sb[b].z : st.kept_base[b];
}

// Budget and idx offset of (sequence b, KV head h); with one budget per
// sequence, hb is NULL.
__host__ __device__ inline int head_budget(const SeqTable &st, const int2 *hb, int Hkv, int b, int h,
                                           const int4 *sb = nullptr) {
  return hb ? hb[b * Hkv + h].x : seq_budget(st, sb, b);
}
__host__ __device__ inline int64_t head_idx_base(const SeqTable &st, const int2 *hb, int Hkv, int b, int h,
                                                 const int4 *sb = nullptr) {
  return (int64_t)seq_idx_base(st, sb, b) + (hb ? hb[b * Hkv + h].y : h * seq_budget(st, sb, b));
}

// Writes n entries of a (budget, offset) table to dst[base ..] (device).
constexpr int kHbChunk = 256;
struct HbChunk {
  int n, base;
  int2 v[kHbChunk];
};
hipError_t launch_set_hb(const HbChunk &c, int2 *dst, hipStream_t s);

// Keys per pipeline stage of the passes for a given number of row tiles.
__host__ __device__ inline int stage_keys(int nw) { return 32 * (nw < 4 ? nw : 4); }
// Dynamic LDS of a pass workgroup.
int pass_lds_bytes(int mode, bool bf16, int head_dim, int rpad, int chunk);

hipError_t launch_pass(int mode, bool bf16, int head_dim, bool w32, const PassArgs &a,
                       const SeqTable &st, hipStream_t s);
// Key-register passes (bf16, up to 128 window rows): keys per workgroup, LDS,
// whether a shape is covered, and the launch of pass 1 (PASS_LSE) or the
// fused pass 2 (PASS_FUSED).
int kr_keys(bool bf16, int head_dim);
int kr_lds_bytes(bool bf16, int head_dim, int rpad);
bool kr_supported(bool bf16, int head_dim, int rpad);
hipError_t launch_krpass(int mode, bool bf16, int head_dim, bool w32, const PassArgs &a,
                         const SeqTable &st, hipStream_t s);
// Streaming pass 2 of one layer (a2) with streaming pass 1 of the next (a1).
hipError_t launch_pass_dual(bool bf16, int head_dim, bool w32, const PassArgs &a2, const PassArgs &a1,
                            const SeqTable &st, hipStream_t s);
// Pass 2 of one layer (a2) with pass 1 of the next layer (a1) in one launch.
hipError_t launch_krdual(bool bf16, int head_dim, bool w32, const PassArgs &a2, const PassArgs &a1,
                         const SeqTable &st, hipStream_t s);
// Single-read pass (bf16, up to 128 window rows): one launch per layer that
// reads K once; needs a.sync (zeroed) and every chunk of the sequence's
// groups resident at once (see single_resident_blocks).
hipError_t launch_single(int head_dim, bool w32, const PassArgs &a, const SeqTable &st, hipStream_t s);
// Workgroups of the single-read pass the device holds at once (0 if unknown).
int single_resident_blocks(int head_dim, int rpad);
int single_lds_bytes(int head_dim, int rpad);
// LDS a select workgroup needs (static + dynamic) for sequences up to max_len.
size_t select_lds_bytes(int mode, int max_len);
hipError_t launch_select(int mode, int max_len, const SelArgs &a, const SeqTable &st,
                         hipStream_t s);
hipError_t launch_elem(const ElemArgs &a, const SeqTable &st, hipStream_t s);
hipError_t launch_lse_merge(const PassArgs &a, const SeqTable &st, hipStream_t s);
hipError_t launch_segcal(const SegArgs &a, const SeqTable &st, hipStream_t s);
// Launches with work of two or three layers of a prompt: the calibration of
// g's layer with the previous layer's candidate lists (gp, may be NULL) and
// the next layer's row normalisers (m, may be NULL); the scores of g's layer
// with the previous layer's final top-K and compaction (gp, may be NULL).
hipError_t launch_sel_a(const SegArgs &g, const SegArgs *gp, const PassArgs *m, const SeqTable &st,
                       hipStream_t s);
hipError_t launch_sel_b(const SegArgs &g, const SegArgs *gp, const SeqTable &st, int max_budget,
                        hipStream_t s);
// LDS of a k_sel_b workgroup (static of both jobs plus the row table).
size_t sel_b_lds_bytes(int max_budget, int window);
hipError_t launch_segscore(const SegArgs &a, const SeqTable &st, hipStream_t s);
hipError_t launch_segcand(const SegArgs &a, const SeqTable &st, hipStream_t s);
// LDS of the final workgroup for budgets up to max_budget.
size_t final_lds_bytes(int max_budget, int window);
size_t alloc_lds_bytes(int hkv);
hipError_t launch_alloc(const AllocArgs &a, const SeqTable &st, hipStream_t s);
hipError_t launch_segfinal(const SegArgs &a, const SeqTable &st, int max_budget, hipStream_t s);
hipError_t launch_compact(const CompactArgs &a, const SeqTable &st, hipStream_t s);
hipError_t launch_zero(unsigned *p, int64_t n, hipStream_t s);
// Device address of the static scratch on the current device (looked up
// once per device); kStaticScratchBytes long.
hipError_t static_scratch(void **ptr);

}  // namespace bacon
