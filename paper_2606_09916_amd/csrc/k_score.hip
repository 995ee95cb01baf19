// Rule score of Eq. 3 over the candidate set A of every session.
//
// The softmax of each memory row runs over all candidates, so the score needs the
// row normaliser before any position can be summed:
//   pass A  (k_score_stats) per (session, tile of positions, unit = (layer, KV head)):
//           logits of the unit's R memory rows against the tile's keys, reduced to a
//           per-tile (max, sum exp) of every row;
//   lse     (k_score_lse)   per row: combine the tiles into (max, 1/Z);
//   pass B  (k_score_rule)  per (session, tile, layer): logits again, p = exp(x - max)/Z,
//           summed over the layer's KV heads and rows;
//   finish  (k_score_finish) per position: sum of the per-layer partials.
// Keys are read through the slot map; dead and forced positions never enter a softmax.
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

__device__ __forceinline__ bool is_forced(const ikv_session &s, int j) {
  return j < s.pi || (j >= s.qs && j < s.qe);
}

template <typename T, int D>
__device__ __forceinline__ void load_row(const T *__restrict__ p, float (&kr)[D]) {
#pragma unroll
  for (int d = 0; d < D; d += 8) load8(p + d, kr + d);
}

template <int D>
__device__ __forceinline__ float dot_lds(const float *__restrict__ m, const float (&kr)[D]) {
  float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
  for (int d = 0; d < D; d += 4) {
    const float4 v = *reinterpret_cast<const float4 *>(m + d);
    a0 = fmaf(v.x, kr[d], a0);
    a1 = fmaf(v.y, kr[d + 1], a1);
    a2 = fmaf(v.z, kr[d + 2], a2);
    a3 = fmaf(v.w, kr[d + 3], a3);
  }
  return (a0 + a1) + (a2 + a3);
}

// ------------------------------------------------------------------ pass A
template <typename T, int D>
__global__ void __launch_bounds__(256) k_score_stats(const T *__restrict__ kpool, int64_t num_slots, int L, int Hkv,
                                                     int dead, const ikv_session *__restrict__ sess,
                                                     const int32_t *__restrict__ slot_maps,
                                                     const float *__restrict__ M, float *__restrict__ ws,
                                                     bool resid) {
  constexpr int RC = 32;                   // memory rows per LDS chunk
  constexpr int XS = SCORE_TILE + 4;       // logit stash row stride
  __shared__ float Ms[RC][D];
  __shared__ float xs[RC][XS];
  const int b = blockIdx.z;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int tile = blockIdx.x;
  const int j0 = tile * SCORE_TILE;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  const int u = blockIdx.y, l = u / Hkv, h = u - l * Hkv;
  const int t = threadIdx.x, j = j0 + t;
  const int32_t *S = slot_maps + s.slot_off;
  bool cand = false;
  int slot = 0;
  if (j < s.N) {
    slot = S[j];
    cand = slot != dead && !is_forced(s, j);
  }
  float kr[D];
  if (cand) {
    load_row<T, D>(kpool + ((int64_t(l) * num_slots + slot) * Hkv + h) * D, kr);
  } else {
#pragma unroll
    for (int d = 0; d < D; ++d) kr[d] = 0.f;
  }
  const float scale = 1.0f / sqrtf(float(D));
  const int64_t tiles = cdiv(s.N, SCORE_TILE);
  float *part = ws + score_offset(sess, b, L, units, D, resid, false);
  const float *Mu = M + s.mem_off + int64_t(u) * s.R * D;

  for (int r0 = 0; r0 < s.R; r0 += RC) {
    const int nr = min(RC, s.R - r0);
    for (int e = t; e < RC * D; e += 256) {
      const int r = e / D, d = e - r * D;
      Ms[r][d] = r < nr ? Mu[int64_t(r0 + r) * D + d] : 0.f;
    }
    __syncthreads();
    for (int r = 0; r < nr; ++r) {
      const float x = dot_lds<D>(&Ms[r][0], kr) * scale;
      xs[r][t] = cand ? x : -INFINITY;
    }
    __syncthreads();
    {
      const int r = t >> 3, q = t & 7;
      float m = -INFINITY;
      for (int i = q; i < SCORE_TILE; i += 8) m = fmaxf(m, xs[r][i]);
      float z = 0.f;
      if (m != -INFINITY)
        for (int i = q; i < SCORE_TILE; i += 8) z += __expf(xs[r][i] - m);
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) {
        const float m2 = __shfl_xor(m, o, WAVE);
        const float z2 = __shfl_xor(z, o, WAVE);
        const float mm = fmaxf(m, m2);
        const float a = (m == -INFINITY) ? 0.f : z * __expf(m - mm);
        const float c = (m2 == -INFINITY) ? 0.f : z2 * __expf(m2 - mm);
        m = mm;
        z = a + c;
      }
      if (q == 0 && r < nr) {
        float *p = part + ((int64_t(u) * s.R + r0 + r) * tiles + tile) * 2;
        p[0] = m;
        p[1] = z;
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ row normalisers
__global__ void __launch_bounds__(256) k_score_lse(const ikv_session *__restrict__ sess, float *__restrict__ ws, int L,
                                                   int units, int D, bool resid) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= units * s.R) return;
  float *base = ws + score_offset(sess, b, L, units, D, resid, false);
  const ScoreSizes z = score_sizes(s, L, units, D, resid, false);
  const int64_t tiles = cdiv(s.N, SCORE_TILE);
  const float *p = base + z.off_part() + int64_t(i) * tiles * 2;
  float m = -INFINITY;
  for (int64_t k = 0; k < tiles; ++k) m = fmaxf(m, p[2 * k]);
  double zs = 0.0;
  if (m != -INFINITY)
    for (int64_t k = 0; k < tiles; ++k)
      if (p[2 * k] != -INFINITY) zs += double(p[2 * k + 1]) * double(expf(p[2 * k] - m));
  float *lse = base + z.off_lse();
  lse[2 * i] = m;
  lse[2 * i + 1] = zs > 0.0 ? float(1.0 / zs) : 0.f;
}

// ------------------------------------------------------------------ pass B
template <typename T, int D>
__global__ void __launch_bounds__(256) k_score_rule(const T *__restrict__ kpool, int64_t num_slots, int L, int Hkv,
                                                    int dead, const ikv_session *__restrict__ sess,
                                                    const int32_t *__restrict__ slot_maps,
                                                    const float *__restrict__ M, float *__restrict__ ws,
                                                    bool resid) {
  constexpr int RC = 64;
  __shared__ float Ms[RC][D];
  __shared__ float st[RC][2];
  const int b = blockIdx.z;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int j0 = blockIdx.x * SCORE_TILE;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  const int l = blockIdx.y;
  const int t = threadIdx.x, j = j0 + t;
  const int32_t *S = slot_maps + s.slot_off;
  bool cand = false;
  int slot = 0;
  if (j < s.N) {
    slot = S[j];
    cand = slot != dead && !is_forced(s, j);
  }
  const float scale = 1.0f / sqrtf(float(D));
  float *base = ws + score_offset(sess, b, L, units, D, resid, false);
  const ScoreSizes z = score_sizes(s, L, units, D, resid, false);
  const float *lse = base + z.off_lse();
  float *rulep = base + z.off_rulep();
  double acc = 0.0;
  float kr[D];
  for (int h = 0; h < Hkv; ++h) {
    const int u = l * Hkv + h;
    if (cand) {
      load_row<T, D>(kpool + ((int64_t(l) * num_slots + slot) * Hkv + h) * D, kr);
    } else {
#pragma unroll
      for (int d = 0; d < D; ++d) kr[d] = 0.f;
    }
    const float *Mu = M + s.mem_off + int64_t(u) * s.R * D;
    for (int r0 = 0; r0 < s.R; r0 += RC) {
      const int nr = min(RC, s.R - r0);
      for (int e = t; e < RC * D; e += 256) {
        const int r = e / D, d = e - r * D;
        Ms[r][d] = r < nr ? Mu[int64_t(r0 + r) * D + d] : 0.f;
      }
      if (t < RC) {
        st[t][0] = t < nr ? lse[(int64_t(u) * s.R + r0 + t) * 2] : 0.f;
        st[t][1] = t < nr ? lse[(int64_t(u) * s.R + r0 + t) * 2 + 1] : 0.f;
      }
      __syncthreads();
      float a = 0.f;
      for (int r = 0; r < nr; ++r) {
        const float x = dot_lds<D>(&Ms[r][0], kr) * scale;
        a += __expf(x - st[r][0]) * st[r][1];
      }
      acc += double(a);
      __syncthreads();
    }
  }
  if (j < s.N) rulep[int64_t(l) * s.N + j] = cand ? float(acc) : 0.f;
}

// ------------------------------------------------------------------ finish
__global__ void __launch_bounds__(256) k_score_finish(const ikv_session *__restrict__ sess,
                                                      const int32_t *__restrict__ slot_maps, int dead,
                                                      float *__restrict__ scores, const float *__restrict__ ws,
                                                      int L, int units, int D, bool resid) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= s.N) return;
  float *out = scores + s.slot_off;
  if (s.N <= s.C) {
    out[j] = -INFINITY;
    return;
  }
  const int slot = slot_maps[s.slot_off + j];
  if (slot == dead || is_forced(s, j)) {
    out[j] = -INFINITY;
    return;
  }
  const float *base = ws + score_offset(sess, b, L, units, D, resid, false);
  const ScoreSizes z = score_sizes(s, L, units, D, resid, false);
  const float *rulep = base + z.off_rulep();
  double acc = 0.0;
  for (int l = 0; l < L; ++l) acc += double(rulep[int64_t(l) * s.N + j]);
  out[j] = float(acc);
}

// ------------------------------------------------------------------ mean key rows (Eq. 5)
template <typename T, int D>
__global__ void __launch_bounds__(256) k_kbar(const T *__restrict__ kpool, int64_t num_slots, int L, int Hkv,
                                              int dead, const ikv_session *__restrict__ sess,
                                              const int32_t *__restrict__ slot_maps, float *__restrict__ ws) {
  constexpr int TPT = D / 2;          // threads per position, two channels each
  constexpr int TOK = 256 / TPT;
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int t = threadIdx.x;
  const int j = blockIdx.x * TOK + t / TPT;
  if (j >= s.N) return;
  const int d = (t % TPT) * 2;
  const int units = L * Hkv;
  float *base = ws + score_offset(sess, b, L, units, D, true, false);
  const ScoreSizes z = score_sizes(s, L, units, D, true, false);
  float *kbar = base + z.off_kbar();
  const int slot = slot_maps[s.slot_off + j];
  float a0 = 0.f, a1 = 0.f;
  if (slot != dead) {
    for (int l = 0; l < L; ++l) {
      const T *p = kpool + (int64_t(l) * num_slots + slot) * Hkv * D + d;
      for (int h = 0; h < Hkv; ++h) {
        a0 += Store<T>::ld(p + h * D);
        a1 += Store<T>::ld(p + h * D + 1);
      }
    }
  }
  const float inv = 1.0f / float(units);
  kbar[int64_t(j) * D + d] = a0 * inv;
  kbar[int64_t(j) * D + d + 1] = a1 * inv;
}

hipError_t launch_residual(const ScoreArgs &a, hipStream_t st);

template <typename T, int D>
static hipError_t launch_score_t(const ScoreArgs &a, hipStream_t st) {
  const ikv_pool &p = a.pool;
  const int units = p.L * p.Hkv;
  const bool resid = (a.flags & IKV_RESIDUAL) != 0;
  const unsigned tiles = unsigned(cdiv(a.maxN, SCORE_TILE));
  const T *kp = static_cast<const T *>(p.k_pool);
  {
    KTimer kt_("k_score_stats<T, D>", st);
    k_score_stats<T, D><<<dim3(tiles, units, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                                 a.slot_maps, a.M, a.ws, resid);
  }
  {
    KTimer kt_("k_score_lse", st);
    k_score_lse<<<dim3(unsigned(cdiv(int64_t(units) * a.maxR, 256)), a.B), 256, 0, st>>>(a.sess_dev, a.ws, p.L, units,
                                                                                         D, resid);
  }
  {
    KTimer kt_("k_score_rule<T, D>", st);
    k_score_rule<T, D><<<dim3(tiles, p.L, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                              a.slot_maps, a.M, a.ws, resid);
  }
  {
    KTimer kt_("k_score_finish", st);
    k_score_finish<<<dim3(unsigned(cdiv(a.maxN, 256)), a.B), 256, 0, st>>>(a.sess_dev, a.slot_maps, p.dead_slot,
                                                                          a.scores, a.ws, p.L, units, D, resid);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !resid) return e;
  constexpr int TOK = 256 / (D / 2);
  {
    KTimer kt_("k_kbar<T, D>", st);
    k_kbar<T, D><<<dim3(unsigned(cdiv(a.maxN, TOK)), a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                         a.sess_dev, a.slot_maps, a.ws);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_residual(a, st);
}

hipError_t launch_score_mfma(const ScoreArgs &a, hipStream_t st);

hipError_t launch_score(const ScoreArgs &a, hipStream_t st) {
  if (a.mfma) return launch_score_mfma(a, st);
  const bool bf = a.pool.kv_dtype == IKV_BF16;
  if (a.pool.D == 128) return bf ? launch_score_t<uint16_t, 128>(a, st) : launch_score_t<float, 128>(a, st);
  return bf ? launch_score_t<uint16_t, 64>(a, st) : launch_score_t<float, 64>(a, st);
}

}  // namespace ikv
