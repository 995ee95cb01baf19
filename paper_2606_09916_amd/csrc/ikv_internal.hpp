// Internal declarations of the IntentKV HIP library: storage helpers, workspace
// layout (evaluated identically on host and device) and kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ikv.h"
#include "ikv_error.hpp"

namespace ikv {

constexpr int WAVE = 64;

// ---------------------------------------------------------------- tiles
constexpr int SCORE_TILE = 256;     // positions per workgroup in the score passes
constexpr int SCORE_ROWS = 64;      // memory rows per chunk held in LDS
constexpr int RES_TILE = 16;        // candidates per workgroup in the residual head
constexpr int DEC_BLOCK = 64;       // live slots per wave per block in decode
constexpr int HC = 128;             // cross-attention width d_c
constexpr int HC_HEADS = 4;         // cross-attention heads H_c
constexpr int HIDDEN = 256;         // residual MLP hidden width
constexpr int MAX_NQ = 256;         // cross-attention query positions per session
constexpr int MAX_R = 256;          // memory rows per KV head

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline int64_t align64f(int64_t n) { return (n + 63) & ~int64_t(63); }   // floats -> 256 B

// Memory rows per KV head rounded up to whole 16-row MFMA slices.
__host__ __device__ inline int pad16(int R) { return (R + 15) & ~15; }

// Score workspace, per session b (floats, each block 256-byte aligned). Two
// layouts: the MFMA path (D = 128, bf16 pool) and the VALU path.
//   msplit [units][pad16(R)][256 bf16]  memory rows pre-split into bf16 hi + lo, the
//          rows past R zero (MFMA only)
//   part   per-tile (max, sum exp) of every memory row:
//            MFMA [tiles of 64 or 128][units][R][2] (room for tiles of 64),
//            VALU [units][R][tiles of 256][2]
//   lse    [units][R][2]          (max, 1/Z) of every memory row, then (MFMA only)
//          [units][R]             -(max + log2 Z), the seed of the second pass
//   rulep  [L][N]                 per-layer partial rule scores (VALU only)
//   kbar   [N][D]                 mean key row (residual only)
//   kq     [nq][D]                kbar at the live query positions (residual only)
//   kp/vp  [nq][HC]               W_K kq + b_K, W_V kq + b_V (residual only)
//   misc   [MBAR_PARTS][D] + [D] + 64   partial and final mbar, live query count (residual only)
//   fold   folded first-layer weights [HC+HIDDEN][D] as bf16 hi + lo, then the
//          constant terms q0 [HC], h0 [HIDDEN], then the rule column of W_Q and W_1
//          [HC+HIDDEN] (residual on the MFMA path only)
//   qlist  [nq] live query positions (residual only)
//   kvf    K' and V' of up to 64 live query positions as bf16 hi + lo MFMA fragments,
//          zero past the live ones (residual on the MFMA path only)
//   mbp    [units / 2][D] column sums of the memory rows per head pair, the partials
//          of mbar when the unit-major first pass runs (residual on the MFMA path only)
//   clist  the candidate list (MFMA path): chunk c of the launch's chunk size CH keeps its
//          candidate positions in position order at [c CH ...], then the counts per
//          chunk (int32)
//   stash  [units][R][NS] float32 logits (log2 domain) of the one-key-pass form (MFMA,
//          R <= 16), indexed by list slot (entry e of chunk c at c CH + e); row stride
//          NS = stash_stride(N), N rounded up to 128, which holds every slot of a list
//          tile that has an entry
// followed by one shared block: W_Q^T [3D+1][HC], W_1^T [3D+1+HC][HIDDEN], and on the
// MFMA path the cross-attention columns of W_1 as bf16 hi + lo [HIDDEN][HC], columns
// ordered within each 32-wide head as perm32 below.
constexpr int MBAR_PARTS = 64;
constexpr int STASH_MAX_R = 16;     // memory rows up to which the MFMA scorer reads the keys once
constexpr int MFMA_TILE = 128;      // positions per workgroup in the MFMA score passes
constexpr int PART_TILE = 64;       // positions per partial of the position-major first pass

struct ScoreSizes {
  int64_t msplit, part, lse, rulep, kbar, kq, kp, vp, misc, fold, qlist, kvf, mbp, clist, stash;
  int64_t lse_pairs;   // units * R * 2: the (max, 1/Z) pairs at the start of lse
  __host__ __device__ int64_t total() const {
    return msplit + part + lse + rulep + kbar + kq + kp + vp + misc + fold + qlist + kvf + mbp + clist + stash;
  }
  __host__ __device__ int64_t off_part() const { return msplit; }
  __host__ __device__ int64_t off_lse() const { return msplit + part; }
  __host__ __device__ int64_t off_rulep() const { return msplit + part + lse; }
  // -(max + log2 Z) per row, after the (max, 1/Z) pairs (MFMA layout only)
  __host__ __device__ int64_t off_nl2() const { return off_lse() + lse_pairs; }
  __host__ __device__ int64_t off_kbar() const { return msplit + part + lse + rulep; }
  __host__ __device__ int64_t off_kq() const { return off_kbar() + kbar; }
  __host__ __device__ int64_t off_kp() const { return off_kq() + kq; }
  __host__ __device__ int64_t off_vp() const { return off_kp() + kp; }
  __host__ __device__ int64_t off_misc() const { return off_vp() + vp; }
  __host__ __device__ int64_t off_fold() const { return off_misc() + misc; }
  __host__ __device__ int64_t off_qlist() const { return off_fold() + fold; }
  __host__ __device__ int64_t off_kvf() const { return off_qlist() + qlist; }
  __host__ __device__ int64_t off_mbp() const { return off_kvf() + kvf; }
  __host__ __device__ int64_t off_clist() const { return off_mbp() + mbp; }
  __host__ __device__ int64_t off_ccount(int N) const { return off_clist() + align64f(int64_t(N) + 1024); }
  __host__ __device__ int64_t off_stash() const { return off_clist() + clist; }
};

// Floats of the folded first-layer weights of one session (bf16 hi + lo, then q0, h0,
// then the rule column).
__host__ __device__ inline int64_t fold_floats(int D) { return int64_t(HC + HIDDEN) * D + 2 * (HC + HIDDEN); }

// Residual cross-attention fragments: K' and V' of RES_KEYS live query positions.
constexpr int RES_KEYS = 64;
constexpr int KVF_BF16 = 2 * HC_HEADS * 4 * 2 * 64 * 8;       // K' then V', 16 KB bf16 each
// Within a 32-wide block, the channel (or key) that MFMA k index 8 g + e stands for:
// lane group g of a 16x16 output block holds rows 4 g .. 4 g + 3 of the block, so the
// two 16-row halves of a 32-wide block give it 4 g + e and 16 + 4 g + e - 4.
__host__ __device__ inline int perm32(int g, int e) { return e < 4 ? 4 * g + e : 16 + 4 * g + (e - 4); }
// and its inverse: channel c of a 32-wide block -> k index 8 g + e
__host__ __device__ inline int perm32_inv(int c) {
  return c < 16 ? 8 * (c >> 2) + (c & 3) : 8 * ((c - 16) >> 2) + 4 + ((c - 16) & 3);
}

__host__ __device__ inline int64_t stash_stride(int N) { return cdiv(int64_t(N), 128) * 128; }

__host__ __device__ inline ScoreSizes score_sizes(const ikv_session &s, int L, int units, int D, bool resid,
                                                  bool mfma) {
  ScoreSizes z;
  z.msplit = mfma ? align64f(int64_t(units) * pad16(s.R) * 128) : 0;
  // MFMA: 64-position partials, or one per 128-entry list tile (at most N / 128 + 8 of
  // them for chunks of up to 1024 positions)
  z.part = mfma ? align64f((cdiv(s.N, PART_TILE) + 8) * units * s.R * 2)
                : align64f(int64_t(units) * s.R * cdiv(s.N, SCORE_TILE) * 2);
  z.lse = align64f(int64_t(units) * s.R * (mfma ? 3 : 2));
  z.lse_pairs = int64_t(units) * s.R * 2;
  z.rulep = mfma ? 0 : align64f(int64_t(L) * s.N);
  z.kbar = resid ? align64f(int64_t(s.N) * D) : 0;
  z.kq = resid ? align64f(int64_t(s.nq) * D) : 0;
  z.kp = resid ? align64f(int64_t(s.nq) * HC) : 0;
  z.vp = z.kp;
  z.misc = resid ? align64f(int64_t(MBAR_PARTS + 1) * D + 64) : 0;
  z.fold = resid && mfma ? align64f(fold_floats(D)) : 0;
  z.qlist = resid ? align64f(s.nq) : 0;
  z.kvf = resid && mfma ? align64f(KVF_BF16 / 2) : 0;
  z.mbp = resid && mfma ? align64f(int64_t(units / 2) * D) : 0;
  z.clist = mfma ? align64f(int64_t(s.N) + 1024) + align64f(cdiv(s.N, 128) + 1) : 0;
  z.stash = mfma && s.R <= STASH_MAX_R ? int64_t(units) * s.R * stash_stride(s.N) : 0;
  return z;
}

// Offset (floats) of session b's score block: the sum of the blocks before it.
__host__ __device__ inline int64_t score_offset(const ikv_session *sess, int b, int L, int units, int D,
                                                bool resid, bool mfma) {
  int64_t o = 0;
  for (int i = 0; i < b; ++i) o += score_sizes(sess[i], L, units, D, resid, mfma).total();
  return o;
}

__host__ __device__ inline int64_t score_shared_floats(int D) {
  return align64f(int64_t(3 * D + 1) * HC) + align64f(int64_t(3 * D + 1 + HC) * HIDDEN) +
         align64f(int64_t(HIDDEN) * HC);
}

// Positions per chunk of the unit-major first pass and of the candidate list of the
// matrix-core path: about nine rounds of two workgroups per CU at the largest sizes,
// whole 128-position multiples (the second pass and the residual head take the list in
// tiles of 128).
inline int stats_chunk(int maxN, int head_pairs) {
  int64_t c = cdiv(cdiv(int64_t(maxN) * head_pairs, 4608), 128) * 128;
  c = c < 128 ? 128 : (c > 1024 ? 1024 : c);
  return int(c);
}

// Redirect workspace: two slot bitsets (kept slots, freed slots) per session.
__host__ __device__ inline int64_t bitset_words(int64_t num_slots) { return align64f(cdiv(num_slots, 32)); }

// Decode workspace: per (session, layer, query head, split) the partial (m, l, o[D]),
// stored as all the o rows ([part][D]) followed by all the (m, l) pairs ([part][2]).
__host__ __device__ inline int64_t decode_part_floats(int D) { return D + 2; }

// ---------------------------------------------------------------- storage
__device__ __forceinline__ float bf16_bits_to_float(uint16_t u) { return __uint_as_float(uint32_t(u) << 16); }

__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);   // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

template <typename T> struct Store;
template <> struct Store<uint16_t> {
  static __device__ __forceinline__ float ld(const uint16_t *p) { return bf16_bits_to_float(*p); }
  static __device__ __forceinline__ uint16_t from(float f) { return float_to_bf16_bits(f); }
};
template <> struct Store<float> {
  static __device__ __forceinline__ float ld(const float *p) { return *p; }
  static __device__ __forceinline__ float from(float f) { return f; }
};

// 8 consecutive elements -> float
__device__ __forceinline__ void load8(const uint16_t *p, float *o) {
  uint4 v = *reinterpret_cast<const uint4 *>(p);
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = __uint_as_float(w[i] << 16);
    o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const float *p, float *o) {
  float4 a = *reinterpret_cast<const float4 *>(p);
  float4 b = *reinterpret_cast<const float4 *>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}

// ---------------------------------------------------------------- wave reductions
// Sum / max over the 64 lanes by DPP row operations (VALU rate, no LDS round trip):
// pairs within quads, half rows, rows, then the row broadcasts leave the total in
// lane 63, which every lane reads back. Every lane of the wave must be active.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ float dpp_f(float old, float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old), __builtin_bit_cast(int, v),
                                                                CTRL, ROW_MASK, 0xf, false));
}
__device__ __forceinline__ float lane63(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(0.f, v);          // quad_perm [1,0,3,2]
  v += dpp_f<0x4E>(0.f, v);          // quad_perm [2,3,0,1]
  v += dpp_f<0x141>(0.f, v);         // row_half_mirror
  v += dpp_f<0x140>(0.f, v);         // row_mirror
  v += dpp_f<0x142, 0xa>(0.f, v);    // row_bcast:15 into rows 1 and 3
  v += dpp_f<0x143, 0xc>(0.f, v);    // row_bcast:31 into rows 2 and 3
  return lane63(v);
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x4E>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x141>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x140>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x142, 0xa>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x143, 0xc>(-INFINITY, v));
  return lane63(v);
}

// ---------------------------------------------------------------- launchers
struct ScoreArgs {
  ikv_pool pool;
  const ikv_session *sess_host;
  const ikv_session *sess_dev;
  int B;
  const int32_t *slot_maps;
  const float *M;
  const int32_t *qpos;
  const float *residual;
  uint32_t flags;
  float *scores;
  float *ws;           // session blocks, then the shared block
  float *ws_shared;
  int maxN, maxR, minR, maxNq;
  int64_t total_positions;   // max over sessions of slot_off + N: the row stride of the per-unit masses
  bool mfma;           // MFMA score passes (D = 128, bf16 pool)
  bool stats;          // the unit-major first pass (MFMA, R <= 64, even Hkv, a layer under 4 GB)
  bool mfma_resid;     // MFMA residual head (MFMA passes and every nq <= 64)
  bool stash;          // one key pass with a logit stash (MFMA, every R <= 16, no IKV_POOL7)
  int fused_tiles;     // > 0: one key pass with the normaliser exchange (k_score_fused), on this many tiles
  uint64_t *xch;       // its exchange area (after the shared block)
};

// The one-key-pass form at 16 < R <= 64 (one session whose list tiles fit on the device
// at once): its workgroup count, 0 where it does not apply; and the floats of its
// exchange area, which follows the score workspace's shared block (0 where it does not
// apply). It is switched off (fused_tiles returns 0): on some calls one row normaliser
// came out wrong, and the cause is not found.
int fused_tiles(const ikv_pool &p, const ikv_session *s, int B, uint32_t flags);
int64_t fused_exchange_floats(const ikv_pool &p, const ikv_session *s, int B, uint32_t flags);

// Opt-in per-kernel timing (ikv_timing in the C ABI): every launch site holds a
// KTimer, which, while timing is on, records a HIP event pair around its launch.
struct KTimer {
  int idx;
  hipStream_t st;
  KTimer(const char *name, hipStream_t stream);
  ~KTimer();
};

hipError_t launch_init_dead_slot(const ikv_pool &pool, hipStream_t st);
hipError_t launch_qm_update(const ikv_pool &pool, const ikv_session *sess_dev, int B, int max_rows,
                            float *M, const void *q_span, float decay, hipStream_t st);
hipError_t launch_score(const ScoreArgs &a, hipStream_t st);
// may_alloc: the call may allocate the pinned host fault word on first use (false on
// the allocation-free entry point, which reports through the word only if it exists).
hipError_t launch_select(const ikv_session *sess_host, const ikv_session *sess_dev, int B, int maxN,
                         const int32_t *slot_maps, int32_t dead, const float *scores, uint8_t *keep,
                         int32_t *n_keep, float *tau, uint32_t *ws, int64_t total_positions, hipStream_t st,
                         bool may_alloc);
// Device address of the allocation-free selection's static scratch on the current
// device (IKV_SELECT_STATIC_MAX_BYTES), resolved on the first call per device.
hipError_t select_static_scratch(uint32_t **ptr);
size_t select_workspace_bytes(const ikv_session *sess, int B, int64_t total_positions);
hipError_t launch_redirect(const ikv_session *sess_dev, int B, int64_t num_slots, int32_t *slot_maps,
                           int32_t dead, const uint8_t *keep, int32_t *freed, int32_t *n_freed,
                           int32_t *live, int32_t *n_live, uint32_t *ws, hipStream_t st);
hipError_t launch_decode(const ikv_pool &pool, const ikv_session *sess_dev, int B, int splits,
                         const void *q, const int32_t *live, const int32_t *n_live, void *out,
                         float *ws, hipStream_t st);

hipError_t launch_compact(const ikv_pool &pool, const ikv_session *sess_dev, int B, int maxN,
                          const int32_t *slot_maps, const uint8_t *keep, const int32_t *dst, double base,
                          int32_t *n_keep, int32_t *pos_list, hipStream_t st);

// Key splits of the prefill attention (one workgroup per layer, KV head, session and
// split of the keys): about nine rounds of workgroups on the 256 CUs (one 8-wave
// workgroup per CU), at most 16 splits and no more than the 64-key tiles of the
// longest session (history bound N plus the span).
inline int prefill_splits(int L, int Hkv, int B, int64_t max_keys) {
  const int64_t units = int64_t(L) * Hkv * (B < 1 ? 1 : B);
  int64_t s = (2304 + units / 2) / units;
  const int64_t tiles = (max_keys + 63) / 64;
  s = s > tiles ? tiles : s;
  return int(s < 1 ? 1 : (s > 16 ? 16 : s));
}
// Prefill workspace: the per-layer parts of the span's mean key rows (span tokens x L x
// D floats); with more than one split, then the split state of the attention, 256 query
// rows per (session, layer, KV head, split): the output rows [part][256][D], then their
// (max, sum) pairs [part][256][2].
inline int64_t prefill_part_floats(int L, int Hkv, int B, int splits, int D) {
  return splits > 1 ? int64_t(B) * L * Hkv * splits * 256 * (D + 2) : 0;
}

hipError_t launch_prefill(const ikv_pool &pool, const ikv_session *sess_dev, int B, int max_n, int splits,
                          const int32_t *slot_maps, const void *q_raw, const void *k_raw, const void *v_raw,
                          const int32_t *hist, const int32_t *n_hist, double base, float decay, float *M,
                          void *q_out, void *out, float *kq, float *ws, int64_t kq_floats, hipStream_t st);

int64_t decode_units(const ikv_pool &p, int B);
int decode_splits(int live_bound, int64_t units);

// A word of pinned host memory that kernels set (system scope) to report a fault the
// host cannot see otherwise (a grid barrier that gave up). Allocated on first use and
// kept for the life of the process; nullptr if the allocation failed. take_host_fault()
// returns whether it was set and clears it.
uint32_t *host_fault_word();
uint32_t *host_fault_word_if_any();   // the word if it exists, never allocating
bool take_host_fault();

}  // namespace ikv
