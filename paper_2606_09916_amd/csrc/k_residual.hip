// Residual head of Eq. 4 with the features of Eq. 5 and the cross-attention of Eq. 6:
//   phi_j = [kbar_j, mbar, kbar_j * mbar, rule_j]
//   c_j   = 4-head attention (width 128, head width 32) of W_Q phi_j + b_Q over the
//           keys W_K kq + b_K and values W_V kq + b_V, kq = kbar at the live query
//           positions; c_j = 0 when the ablation flag is set or no query position is live
//   s_j   = rule_j + clip(alpha, -5, 5) * (w_2 . GELU(W_1 [phi_j ; c_j] + b_1) + b_2)
// All arithmetic is float32. The rule scores arrive in `scores` and are overwritten.
#include <math.h>

#include "ikv_internal.hpp"
#include "res_setup.hpp"

namespace ikv {

int64_t residual_floats(int D) { return ResLayout(D).total; }

// W_Q^T [F][HC] and W_1^T [F+HC][HIDDEN] so that consecutive threads read consecutive
// outputs, and the cross-attention columns of W_1 as bf16 hi [HIDDEN][HC] then lo,
// each 32-wide head block in the MFMA k order of perm32.
__global__ void k_res_transpose(const float *__restrict__ blob, float *__restrict__ shared, int D) {
  const ResLayout lay(D);
  const int64_t F = 3 * D + 1;
  const int64_t nq = F * HC, n1 = (F + HC) * HIDDEN, nc = int64_t(HIDDEN) * HC;
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  float *wqT = shared;
  float *w1T = shared + align64f(F * HC);
  uint16_t *w1c = reinterpret_cast<uint16_t *>(w1T + align64f((F + HC) * HIDDEN));
  if (i < nq) {
    const int64_t in = i / HC, o = i - in * HC;
    wqT[i] = blob[lay.WQ + o * F + in];
  } else if (i < nq + n1) {
    const int64_t k = i - nq;
    const int64_t in = k / HIDDEN, o = k - in * HIDDEN;
    w1T[k] = blob[lay.W1 + o * (F + HC) + in];
  } else if (i < nq + n1 + nc) {
    const int64_t k = i - nq - n1;
    const int64_t o = k / HC, c = k - o * HC;
    const float v = blob[lay.W1 + o * (F + HC) + F + c];
    const uint16_t hi = float_to_bf16_bits(v);
    const int64_t at = o * HC + (c & ~int64_t(31)) + perm32_inv(int(c & 31));
    w1c[at] = hi;
    w1c[nc + at] = float_to_bf16_bits(v - bf16_bits_to_float(hi));
  }
}

// Partial column sums of the memory rows: part p sums rows [p*rows/P, (p+1)*rows/P).
template <int D>
__global__ void __launch_bounds__(256) k_mbar_part(const ikv_session *__restrict__ sess, const float *__restrict__ M,
                                                   float *__restrict__ ws, int L, int Hkv, bool mfma) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const int64_t rows = int64_t(units) * s.R;
  const int p = blockIdx.x;
  const int64_t r0 = rows * p / MBAR_PARTS, r1 = rows * (p + 1) / MBAR_PARTS;
  __shared__ float red[256 / D][D];
  const int d = threadIdx.x % D, g = threadIdx.x / D;
  constexpr int NG = 256 / D;
  float a = 0.f;
  for (int64_t r = r0 + g; r < r1; r += NG) a += M[s.mem_off + r * D + d];
  red[g][d] = a;
  __syncthreads();
  if (g == 0) {
    float t = 0.f;
    for (int k = 0; k < NG; ++k) t += red[k][d];
    const ScoreSizes z = score_sizes(s, L, units, D, true, mfma);
    float *misc = ws + score_offset(sess, b, L, units, D, true, mfma) + z.off_misc();
    misc[int64_t(p) * D + d] = t;
  }
}

// Per session: mbar and the live query positions (res_setup_body), one workgroup each.
template <int D>
__global__ void __launch_bounds__(256) k_res_setup(const ikv_session *__restrict__ sess,
                                                   const int32_t *__restrict__ slot_maps,
                                                   const int32_t *__restrict__ qpos, int dead, float *__restrict__ ws,
                                                   int L, int Hkv, bool mfma, bool pairs) {
  res_setup_body<D>(sess, int(blockIdx.x), slot_maps, qpos, dead, ws, L, Hkv, mfma, pairs);
}

// kq on the matrix-core path, where the second pass keeps kbar at the candidates only
// (a live query position in the query span is never one): row i of the kq block is the
// mean over the L Hkv units of the bf16 key row of the i-th live query position, summed
// layer-major in float32 and scaled by 1 / (L Hkv) as the second pass does. One
// workgroup per live row, thread = channel.
template <int D>
__global__ void __launch_bounds__(D) k_res_kq(const ikv_session *__restrict__ sess, const uint16_t *__restrict__ kpool,
                                              int64_t num_slots, int L, int Hkv,
                                              const int32_t *__restrict__ slot_maps, float *__restrict__ ws) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const ScoreSizes z = score_sizes(s, L, units, D, true, true);
  float *base = ws + score_offset(sess, b, L, units, D, true, true);
  const int n = reinterpret_cast<const int *>(base + z.off_misc() + int64_t(MBAR_PARTS) * D)[D];
  const int i = blockIdx.x;
  if (i >= n) return;
  const int q = reinterpret_cast<const int *>(base + z.off_qlist())[i];
  const int64_t slot = slot_maps[s.slot_off + q];
  const int d = threadIdx.x;
  float a = 0.f;
  for (int u = 0; u < units; ++u) {
    const int l = u / Hkv, h = u - l * Hkv;
    a += bf16_bits_to_float(kpool[((int64_t(l) * num_slots + slot) * Hkv + h) * D + d]);
  }
  base[z.off_kq() + int64_t(i) * D + d] = a * (1.0f / float(units));
}

// K' = W_K kq + b_K and V' = W_V kq + b_V for four live query rows per workgroup,
// kq = kbar at the live query positions (from the second pass; on the matrix-core path
// the kq block of k_res_kq, row i for the i-th live row).
template <int D>
__device__ __forceinline__ void res_kv_body(int bx, const ikv_session *__restrict__ sess, const float *__restrict__ blob,
                                            float *__restrict__ ws, int L, int Hkv, bool mfma) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const ResLayout lay(D);
  const ScoreSizes z = score_sizes(s, L, units, D, true, mfma);
  float *base = ws + score_offset(sess, b, L, units, D, true, mfma);
  const float *kbar = base + (mfma ? z.off_kq() : z.off_kbar());
  float *kp = base + z.off_kp();
  float *vp = base + z.off_vp();
  const int n = reinterpret_cast<const int *>(base + z.off_misc() + int64_t(MBAR_PARTS) * D)[D];
  const int *qlist = reinterpret_cast<const int *>(base + z.off_qlist());
  const int i0 = bx * 4;
  if (i0 >= n) return;
  __shared__ float kq[4][D];
  const int t = threadIdx.x;
  for (int e = t; e < 4 * D; e += 256) {
    const int r = e / D, d = e - r * D;
    const int i = min(i0 + r, n - 1);                  // a live row stands in past n
    const float v = kbar[int64_t(mfma ? i : qlist[i]) * D + d];
    kq[r][d] = (i0 + r < n) ? v : 0.f;
  }
  __syncthreads();
  const int o = t & (HC - 1);
  const bool isv = t >= HC;
  const float *W = blob + (isv ? lay.WV : lay.WK) + int64_t(o) * D;
  const float bias = blob[(isv ? lay.bV : lay.bK) + o];
  float a[4] = {bias, bias, bias, bias};
  constexpr int WB = 64;                              // weights in flight per thread
#pragma unroll 1
  for (int d0 = 0; d0 < D; d0 += WB) {
    float wv[WB];
#pragma unroll
    for (int d = 0; d < WB; ++d) wv[d] = W[d0 + d];
#pragma unroll
    for (int d = 0; d < WB; ++d)
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = fmaf(wv[d], kq[r][d0 + d], a[r]);
  }
  float *dst = isv ? vp : kp;
#pragma unroll
  for (int r = 0; r < 4; ++r)
    if (i0 + r < n) dst[int64_t(i0 + r) * HC + o] = a[r];
}

template <int D>
__global__ void __launch_bounds__(256) k_res_kv(const ikv_session *__restrict__ sess, const float *__restrict__ blob,
                                                float *__restrict__ ws, int L, int Hkv, bool mfma) {
  res_kv_body<D>(int(blockIdx.x), sess, blob, ws, L, Hkv, mfma);
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

template <int D>
__global__ void __launch_bounds__(256) k_residual(const ikv_session *__restrict__ sess,
                                                  const int32_t *__restrict__ slot_maps, int dead,
                                                  float *__restrict__ scores, const float *__restrict__ ws,
                                                  const float *__restrict__ shared, const float *__restrict__ blob,
                                                  int L, int Hkv, bool xattn, bool mfma) {
  constexpr int F = 3 * D + 1;
  constexpr int X = F + HC;
  constexpr int TK = 32;       // candidates per workgroup
  constexpr int KC = 32;       // query keys per LDS chunk
  __shared__ float xT[X][TK];          // [phi ; c] transposed: xT[i][k]
  __shared__ float ql[TK][HC + 4];     // W_Q phi + b_Q
  __shared__ float kvl[2][KC][HC];     // K', V' chunk
  __shared__ float red[4][TK];
  __shared__ int pos[TK];
  __shared__ int any;

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int j0 = blockIdx.x * TK;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  const ResLayout lay(D);
  const ScoreSizes z = score_sizes(s, L, units, D, true, mfma);
  const float *base = ws + score_offset(sess, b, L, units, D, true, mfma);
  const float *kbar = base + z.off_kbar();
  const float *kp = base + z.off_kp();
  const float *vp = base + z.off_vp();
  const float *mbar = base + z.off_misc() + int64_t(MBAR_PARTS) * D;
  const int nql = reinterpret_cast<const int *>(mbar)[D];
  const float *wqT = shared;
  const float *w1T = shared + align64f(int64_t(F) * HC);
  float *out = scores + s.slot_off;
  const int t = threadIdx.x;

  if (t == 0) any = 0;
  __syncthreads();
  if (t < TK) {
    const int j = j0 + t;
    bool c = false;
    if (j < s.N) {
      const int slot = slot_maps[s.slot_off + j];
      c = slot != dead && !(j < s.pi || (j >= s.qs && j < s.qe));
    }
    pos[t] = c ? j : -1;
    if (c) atomicOr(&any, 1);
  }
  __syncthreads();
  if (!any) return;

  // phi
  for (int e = t; e < TK * F; e += 256) {
    const int i = e / TK, k = e - i * TK;
    const int j = pos[k];
    float v = 0.f;
    if (j >= 0) {
      if (i < D) v = kbar[int64_t(j) * D + i];
      else if (i < 2 * D) v = mbar[i - D];
      else if (i < 3 * D) v = kbar[int64_t(j) * D + (i - 2 * D)] * mbar[i - 2 * D];
      else v = out[j];
    }
    xT[i][k] = v;
  }
  __syncthreads();

  // Q = W_Q phi + b_Q : thread -> output o, 16 candidates
  {
    const int o = t & (HC - 1), k0 = (t >> 7) * 16;
    float acc[16];
    const float bq = blob[lay.bQ + o];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = bq;
    for (int i = 0; i < F; ++i) {
      const float w = wqT[int64_t(i) * HC + o];
#pragma unroll
      for (int k = 0; k < 16; k += 4) {
        const float4 xv = *reinterpret_cast<const float4 *>(&xT[i][k0 + k]);
        acc[k] = fmaf(xv.x, w, acc[k]);
        acc[k + 1] = fmaf(xv.y, w, acc[k + 1]);
        acc[k + 2] = fmaf(xv.z, w, acc[k + 2]);
        acc[k + 3] = fmaf(xv.w, w, acc[k + 3]);
      }
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) ql[k0 + k][o] = acc[k];
  }
  __syncthreads();

  // cross-attention: thread -> (candidate k, head hh, half of the head's 32 channels)
  {
    const int k = t >> 3, hh = (t >> 1) & 3, half = t & 1;
    const int c0 = hh * 32 + half * 16;
    float q[16], o[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      q[c] = ql[k][c0 + c];
      o[c] = 0.f;
    }
    float m = -INFINITY, lsum = 0.f;
    const bool on = xattn && nql > 0;
    const float scale = 0.17677669529663688f;   // 1/sqrt(32)
    for (int p0 = 0; on && p0 < nql; p0 += KC) {
      const int np = min(KC, nql - p0);
      __syncthreads();
      for (int e = t; e < KC * HC; e += 256) {
        const int p = e / HC, c = e - p * HC;
        kvl[0][p][c] = p < np ? kp[int64_t(p0 + p) * HC + c] : 0.f;
        kvl[1][p][c] = p < np ? vp[int64_t(p0 + p) * HC + c] : 0.f;
      }
      __syncthreads();
      for (int p = 0; p < np; ++p) {
        float x = 0.f;
#pragma unroll
        for (int c = 0; c < 16; ++c) x = fmaf(q[c], kvl[0][p][c0 + c], x);
        x += __shfl_xor(x, 1, WAVE);
        x *= scale;
        const float mn = fmaxf(m, x);
        const float corr = (m == -INFINITY) ? 0.f : expf(m - mn);
        const float w = expf(x - mn);
        lsum = lsum * corr + w;
#pragma unroll
        for (int c = 0; c < 16; ++c) o[c] = fmaf(w, kvl[1][p][c0 + c], o[c] * corr);
        m = mn;
      }
    }
    const float inv = lsum > 0.f ? 1.0f / lsum : 0.f;
#pragma unroll
    for (int c = 0; c < 16; ++c) xT[F + c0 + c][k] = o[c] * inv;
  }
  __syncthreads();

  // hidden layer: thread -> hidden unit o, all 32 candidates
  {
    const int o = t;
    float acc[TK];
    const float b1 = blob[lay.b1 + o];
#pragma unroll
    for (int k = 0; k < TK; ++k) acc[k] = b1;
    for (int i = 0; i < X; ++i) {
      const float w = w1T[int64_t(i) * HIDDEN + o];
#pragma unroll
      for (int k = 0; k < TK; k += 4) {
        const float4 xv = *reinterpret_cast<const float4 *>(&xT[i][k]);
        acc[k] = fmaf(xv.x, w, acc[k]);
        acc[k + 1] = fmaf(xv.y, w, acc[k + 1]);
        acc[k + 2] = fmaf(xv.z, w, acc[k + 2]);
        acc[k + 3] = fmaf(xv.w, w, acc[k + 3]);
      }
    }
    const float w2 = blob[lay.w2 + o];
    const int wave = t >> 6;
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      const float y = wave_sum(gelu_erf(acc[k]) * w2);
      if ((t & 63) == 0) red[wave][k] = y;
    }
  }
  __syncthreads();
  if (t < TK && pos[t] >= 0) {
    const float alpha = fminf(fmaxf(blob[lay.alpha], -5.0f), 5.0f);
    const float y = ((red[0][t] + red[1][t]) + (red[2][t] + red[3][t])) + blob[lay.b2];
    const int j = pos[t];
    out[j] = out[j] + alpha * y;
  }
}

hipError_t launch_residual_mfma(const ScoreArgs &a, hipStream_t st);

template <int D>
static hipError_t launch_residual_t(const ScoreArgs &a, hipStream_t st) {
  const ikv_pool &p = a.pool;
  const int64_t F = 3 * D + 1;
  const int64_t n = F * HC + (F + HC) * HIDDEN + int64_t(HIDDEN) * HC;
  if (!a.mfma_resid)
    {
      KTimer kt_("k_res_transpose", st);
      k_res_transpose<<<unsigned(cdiv(n, 256)), 256, 0, st>>>(a.residual, a.ws_shared, D);
    }
  if (!a.mfma)   // on the matrix-core path k_msplit leaves the partial sums of mbar
  {
    KTimer kt_("k_mbar_part<D>", st);
    k_mbar_part<D><<<dim3(MBAR_PARTS, a.B), 256, 0, st>>>(a.sess_dev, a.M, a.ws, p.L, p.Hkv, a.mfma);
  }
  if (!a.mfma)   // on the matrix-core path the row-statistics launch did the set-up
    {
      KTimer kt_("k_res_setup<D>", st);
      k_res_setup<D><<<a.B, 256, 0, st>>>(a.sess_dev, a.slot_maps, a.qpos, p.dead_slot, a.ws, p.L, p.Hkv, a.mfma,
                                          a.stats);
    }
  if (a.maxNq > 0 && !a.mfma_resid && a.mfma)
    {
      KTimer kt_("k_res_kq<D>", st);
      k_res_kq<D><<<dim3(unsigned(a.maxNq), a.B), D, 0, st>>>(a.sess_dev, static_cast<const uint16_t *>(p.k_pool),
                                                              p.num_slots, p.L, p.Hkv, a.slot_maps, a.ws);
    }
  if (a.maxNq > 0 && !a.mfma_resid)
    {
      KTimer kt_("k_res_kv<D>", st);
      k_res_kv<D><<<dim3(unsigned(cdiv(a.maxNq, 4)), a.B), 256, 0, st>>>(a.sess_dev, a.residual, a.ws, p.L, p.Hkv,
                                                                         a.mfma);
    }
  // on the matrix-core path the row-statistics launch also folded the first layer and
  // built the K', V' fragments
  if (a.mfma_resid) return launch_residual_mfma(a, st);
  {
    KTimer kt_("k_residual<D>", st);
    k_residual<D><<<dim3(unsigned(cdiv(a.maxN, 32)), a.B), 256, 0, st>>>(
        a.sess_dev, a.slot_maps, p.dead_slot, a.scores, a.ws, a.ws_shared, a.residual, p.L, p.Hkv,
        (a.flags & IKV_NO_XATTN) == 0, a.mfma);
  }
  return hipGetLastError();
}

hipError_t launch_residual(const ScoreArgs &a, hipStream_t st) {
  return a.pool.D == 128 ? launch_residual_t<128>(a, st) : launch_residual_t<64>(a, st);
}

}  // namespace ikv
