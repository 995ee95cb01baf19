// Rule score of Eq. 3 on the matrix cores (bf16 pool, head dimension 128, memory
// rows per KV head a multiple of 16).
//
// The logits x = M . K / sqrt(D) of a unit (layer, KV head) and a tile of 128
// positions form a [128 x R] product with a 128-long contraction. They run as
// v_mfma_f32_16x16x32_bf16 with K (exact in bf16) as the A operand and the memory
// rows as the B operand. Each memory row is pre-split into bf16 hi + lo
// (M' = hi + lo to 2^-18 relative), so two MFMAs per fragment give float32-grade
// logits. log2(e)/sqrt(D) is folded into M', so the softmax uses native exp2.
//
// One workgroup owns 128 positions and walks every unit: the unit's keys are
// staged in LDS with 256-byte coalesced row loads (the next unit's rows are
// fetched into registers while the current one computes), and wave w takes the
// 16-row slices w, w+4, ... of the memory.
//   pass A: per (tile, unit, row) the max and sum of exp2 over the tile's candidates;
//   lse:    per (unit, row) the tiles combine into (max, 1/Z);
//   pass B: p = exp2(x - max) / Z summed over every unit and row, per position, in
//           registers; with the residual head on, the mean key row accumulates from
//           the same LDS tiles.
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int MD = 128;          // head dimension of this path
constexpr int KROW = MD + 8;     // LDS row stride in bf16 (272 B): 16-lane column reads hit 64 distinct banks
constexpr float LOG2E = 1.4426950408889634f;

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// M' = M * log2(e) / sqrt(D) split into bf16 hi and lo. Per (unit, row): four groups
// of 32 channels, each stored as [hi 32 | lo 32].
__global__ void __launch_bounds__(256) k_msplit(const ikv_session *__restrict__ sess, const float *__restrict__ M,
                                                float *__restrict__ ws, int L, int Hkv, bool resid) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= int64_t(units) * s.R * 4) return;
  const int64_t row = i >> 2;
  const int g = int(i & 3);
  const float scale = LOG2E / sqrtf(float(MD));
  const float *src = M + s.mem_off + row * MD + g * 32;
  uint16_t *dst = reinterpret_cast<uint16_t *>(ws + score_offset(sess, b, L, units, MD, resid, true)) + row * 256 +
                  g * 64;
  for (int e = 0; e < 32; ++e) {
    const float v = src[e] * scale;
    const uint16_t hi = float_to_bf16_bits(v);
    dst[e] = hi;
    dst[32 + e] = float_to_bf16_bits(v - bf16_bits_to_float(hi));
  }
}

template <bool PASS_B, bool KBAR>
__global__ void __launch_bounds__(256) k_score_mfma(const uint16_t *__restrict__ kpool, int64_t num_slots, int L,
                                                       int Hkv, int dead, const ikv_session *__restrict__ sess,
                                                       const int32_t *__restrict__ slot_maps, float *__restrict__ ws,
                                                       float *__restrict__ scores, bool resid) {
  __shared__ __align__(16) uint16_t kt[2][MFMA_TILE * KROW];
  __shared__ int slot_s[MFMA_TILE];
  __shared__ int cand_s[MFMA_TILE];
  __shared__ float red[4][MFMA_TILE];

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int tile = blockIdx.x;
  const int j0 = tile * MFMA_TILE;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int R = s.R, nsl = R >> 4;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const uint16_t *msplit = reinterpret_cast<const uint16_t *>(base);
  float *part = base + z.off_part();
  const float *lse = base + z.off_lse();

  if (t < MFMA_TILE) {
    const int j = j0 + t;
    int slot = -1, c = 0;
    if (j < s.N) {
      slot = slot_maps[s.slot_off + j];
      c = slot != dead && !(j < s.pi || (j >= s.qs && j < s.qe));
    }
    slot_s[t] = slot;
    cand_s[t] = c;
  }
  __syncthreads();

  // key-row loader: 16 threads per 256-byte row, rows lr + 16 i
  const int lc = t & 15, lr = t >> 4;
  const int64_t slot_stride = int64_t(Hkv) * MD;
  uint4 pre[8];
  auto fetch = [&](int u) {
    const int l = u / Hkv, h = u - l * Hkv;
    const uint16_t *bl = kpool + int64_t(l) * num_slots * slot_stride + int64_t(h) * MD + lc * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int sl = slot_s[lr + 16 * i];
      pre[i] = sl >= 0 ? *reinterpret_cast<const uint4 *>(bl + int64_t(sl) * slot_stride) : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<uint4 *>(&kt[buf][(lr + 16 * i) * KROW + lc * 8]) = pre[i];
  };

  float racc[8][4];
  float kb[64];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) racc[i][k] = 0.f;
#pragma unroll
  for (int i = 0; i < 64; ++i) kb[i] = 0.f;

  fetch(0);
  stash(0);
  __syncthreads();
  for (int u = 0; u < units; ++u) {
    const int buf = u & 1;
    if (u + 1 < units) fetch(u + 1);
    const uint16_t *kl = kt[buf];
    for (int sl = w; sl < nsl; sl += 4) {
      const int row = sl * 16 + (lane & 15);
      const uint16_t *mp = msplit + (int64_t(u) * R + row) * 256 + (lane >> 4) * 64;
      bf16x8 mh[4], ml[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        mh[ks] = *reinterpret_cast<const bf16x8 *>(mp + ks * 8);
        ml[ks] = *reinterpret_cast<const bf16x8 *>(mp + 32 + ks * 8);
      }
      float mrow = 0.f, iz = 0.f;
      if (PASS_B) {
        mrow = lse[(int64_t(u) * R + row) * 2];
        iz = lse[(int64_t(u) * R + row) * 2 + 1];
      }
      float m = -INFINITY, zs = 0.f;
#pragma unroll
      for (int blk = 0; blk < MFMA_TILE / 16; ++blk) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        const uint16_t *kr = kl + (blk * 16 + (lane & 15)) * KROW + (lane >> 4) * 32;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kr + ks * 8);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, mh[ks], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, ml[ks], acc, 0, 0, 0);
        }
        // acc[i]: position blk*16 + 4*(lane >> 4) + i, memory row `row`
        const int tb = blk * 16 + 4 * (lane >> 4);
        if (!PASS_B) {
          const float x0 = cand_s[tb] ? acc[0] : -INFINITY;
          const float x1 = cand_s[tb + 1] ? acc[1] : -INFINITY;
          const float x2 = cand_s[tb + 2] ? acc[2] : -INFINITY;
          const float x3 = cand_s[tb + 3] ? acc[3] : -INFINITY;
          const float bm = fmaxf(fmaxf(x0, x1), fmaxf(x2, x3));
          if (bm > m) {
            zs *= exp2f(m - bm);
            m = bm;
          }
          if (m != -INFINITY) zs += (exp2f(x0 - m) + exp2f(x1 - m)) + (exp2f(x2 - m) + exp2f(x3 - m));
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (cand_s[tb + i]) racc[blk][i] += exp2f(acc[i] - mrow) * iz;
        }
      }
      if (!PASS_B) {
#pragma unroll
        for (int o = 16; o < 64; o <<= 1) {
          const float m2 = __shfl_xor(m, o, WAVE);
          const float z2 = __shfl_xor(zs, o, WAVE);
          const float mm = fmaxf(m, m2);
          const float a = (m == -INFINITY) ? 0.f : zs * exp2f(m - mm);
          const float c = (m2 == -INFINITY) ? 0.f : z2 * exp2f(m2 - mm);
          m = mm;
          zs = a + c;
        }
        if (lane < 16) {
          float *p = part + ((int64_t(tile) * units + u) * R + row) * 2;
          p[0] = m;
          p[1] = zs;
        }
      }
    }
    if (KBAR) {
      const uint16_t *kr = kl + (32 * w + (lane & 31)) * KROW + (lane >> 5) * 64;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint4 v = *reinterpret_cast<const uint4 *>(kr + 8 * i);
        kb[8 * i + 0] += bf_lo(v.x);
        kb[8 * i + 1] += bf_hi(v.x);
        kb[8 * i + 2] += bf_lo(v.y);
        kb[8 * i + 3] += bf_hi(v.y);
        kb[8 * i + 4] += bf_lo(v.z);
        kb[8 * i + 5] += bf_hi(v.z);
        kb[8 * i + 6] += bf_lo(v.w);
        kb[8 * i + 7] += bf_hi(v.w);
      }
    }
    if (u + 1 < units) stash(buf ^ 1);
    __syncthreads();
  }

  if (PASS_B) {
#pragma unroll
    for (int blk = 0; blk < MFMA_TILE / 16; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = racc[blk][i];
        v += __shfl_xor(v, 1, WAVE);
        v += __shfl_xor(v, 2, WAVE);
        v += __shfl_xor(v, 4, WAVE);
        v += __shfl_xor(v, 8, WAVE);
        if ((lane & 15) == 0) red[w][blk * 16 + 4 * (lane >> 4) + i] = v;
      }
    __syncthreads();
    if (t < MFMA_TILE) {
      const int j = j0 + t;
      if (j < s.N)
        scores[s.slot_off + j] = cand_s[t] ? (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]) : -INFINITY;
    }
  }
  if (KBAR) {
    const int tok = 32 * w + (lane & 31);
    const int j = j0 + tok;
    if (j < s.N) {
      const float inv = 1.0f / float(units);
      float *dst = base + z.off_kbar() + int64_t(j) * MD + (lane >> 5) * 64;
#pragma unroll
      for (int e = 0; e < 64; e += 4)
        *reinterpret_cast<float4 *>(dst + e) = make_float4(kb[e] * inv, kb[e + 1] * inv, kb[e + 2] * inv,
                                                           kb[e + 3] * inv);
    }
  }
}

// Per (unit, row): combine the per-tile statistics into (max, 1/Z), log2 domain.
__global__ void __launch_bounds__(256) k_lse_mfma(const ikv_session *__restrict__ sess, float *__restrict__ ws, int L,
                                                  int Hkv, bool resid) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const int64_t rows = int64_t(units) * s.R;
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= rows) return;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const float *part = base + z.off_part();
  const int64_t tiles = cdiv(s.N, MFMA_TILE);
  float m = -INFINITY;
  for (int64_t k = 0; k < tiles; ++k) m = fmaxf(m, part[(k * rows + i) * 2]);
  double zs = 0.0;
  if (m != -INFINITY)
    for (int64_t k = 0; k < tiles; ++k) {
      const float mk = part[(k * rows + i) * 2];
      if (mk != -INFINITY) zs += double(part[(k * rows + i) * 2 + 1]) * double(exp2f(mk - m));
    }
  float *lse = base + z.off_lse();
  lse[2 * i] = m;
  lse[2 * i + 1] = zs > 0.0 ? float(1.0 / zs) : 0.f;
}

// The gate: sessions with N <= C get -inf everywhere (the passes skip them).
__global__ void k_fill_skipped(const ikv_session *__restrict__ sess, float *__restrict__ scores) {
  const ikv_session s = sess[blockIdx.y];
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (s.N <= s.C && j < s.N) scores[s.slot_off + j] = -INFINITY;
}

hipError_t launch_residual(const ScoreArgs &a, hipStream_t st);

hipError_t launch_score_mfma(const ScoreArgs &a, hipStream_t st) {
  const ikv_pool &p = a.pool;
  const int units = p.L * p.Hkv;
  const bool resid = (a.flags & IKV_RESIDUAL) != 0;
  const unsigned tiles = unsigned(cdiv(a.maxN, MFMA_TILE));
  const uint16_t *kp = static_cast<const uint16_t *>(p.k_pool);
  k_fill_skipped<<<dim3(unsigned(cdiv(a.maxN, 256)), a.B), 256, 0, st>>>(a.sess_dev, a.scores);
  k_msplit<<<dim3(unsigned(cdiv(int64_t(units) * a.maxR * 4, 256)), a.B), 256, 0, st>>>(a.sess_dev, a.M, a.ws, p.L,
                                                                                        p.Hkv, resid);
  k_score_mfma<false, false><<<dim3(tiles, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                               a.slot_maps, a.ws, a.scores, resid);
  k_lse_mfma<<<dim3(unsigned(cdiv(int64_t(units) * a.maxR, 256)), a.B), 256, 0, st>>>(a.sess_dev, a.ws, p.L, p.Hkv,
                                                                                      resid);
  if (resid)
    k_score_mfma<true, true><<<dim3(tiles, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                               a.slot_maps, a.ws, a.scores, resid);
  else
    k_score_mfma<true, false><<<dim3(tiles, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                a.sess_dev, a.slot_maps, a.ws, a.scores, resid);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !resid) return e;
  return launch_residual(a, st);
}

}  // namespace ikv
