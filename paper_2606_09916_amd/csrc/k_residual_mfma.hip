// Residual head of Eq. 4 (features Eq. 5, cross-attention Eq. 6) on the matrix cores,
// for D = 128 and at most 64 live query positions per session.
//
// With mbar folded into the first-layer weights (k_res_fold), one tile of 64
// candidates is a chain of four small products on v_mfma_f32_16x16x32_bf16:
//   1. [Q ; hidden] = kbar . A^T + (q0 ; h0) + (w_Q^r ; w_1^r) rule    (64 x 384, K = 128)
//   2. logits_h = Q_h . K'_h^T / sqrt(32)                                (per head, 64 x 64, K = 32)
//   3. c_h = softmax(logits_h) . V'_h                                    (per head, 64 x 32, K = 64)
//   4. hidden += c . W_1^c^T                                             (64 x 256, K = 128)
// then y = w_2 . GELU(hidden) + b_2 and s = rule + clip(alpha, -5, 5) y.
// Every operand is split into bf16 hi + lo and each product runs as hi.hi + hi.lo +
// lo.hi with float32 accumulation (relative error about 2^-17 per product).
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int RD = 128;          // head dimension of this path
constexpr int RT = 64;           // candidates per workgroup
constexpr int XS = RD + 8;       // LDS row stride (bf16) of 128-wide rows (272 B)
constexpr int PS = 64 + 8;       // LDS row stride (bf16) of 64-wide rows (144 B)
constexpr int RES_MAX_KEYS = 64; // live query positions handled by this path

__device__ __forceinline__ void split_bf16(float v, uint16_t &h, uint16_t &l) {
  h = float_to_bf16_bits(v);
  l = float_to_bf16_bits(v - bf16_bits_to_float(h));
}

__device__ __forceinline__ f32x4 mfma3(const bf16x8 &ah, const bf16x8 &al, const bf16x8 &bh, const bf16x8 &bl,
                                       f32x4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
  return acc;
}

__device__ __forceinline__ bf16x8 ld8(const uint16_t *p) { return *reinterpret_cast<const bf16x8 *>(p); }

__device__ __forceinline__ float gelu_exact(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

__global__ void __launch_bounds__(256) k_residual_mfma(const ikv_session *__restrict__ sess,
                                                       const int32_t *__restrict__ slot_maps, int dead,
                                                       float *__restrict__ scores, const float *__restrict__ ws,
                                                       const float *__restrict__ shared,
                                                       const float *__restrict__ blob, int L, int Hkv, bool xattn) {
  __shared__ __align__(16) uint16_t xs[2][RT * XS];              // kbar, then Q, then c
  __shared__ __align__(16) uint16_t kps[2][RES_MAX_KEYS * XS];   // K' [key][channel]
  __shared__ __align__(16) uint16_t vts[2][RD * PS];             // V'^T [channel][key]
  __shared__ __align__(16) uint16_t ps[2][RT * PS];              // softmax weights of one head
  __shared__ float rule_s[RT];
  __shared__ float red[4][RT];
  __shared__ int pos_s[RT];
  __shared__ int any;

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int j0 = blockIdx.x * RT;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  constexpr int64_t F = 3 * RD + 1;
  const ScoreSizes z = score_sizes(s, L, units, RD, true, true);
  const float *base = ws + score_offset(sess, b, L, units, RD, true, true);
  const float *kbar = base + z.off_kbar();
  const float *kp = base + z.off_kp();
  const float *vp = base + z.off_vp();
  const float *mbar = base + z.off_misc() + int64_t(MBAR_PARTS) * RD;
  const int nql = reinterpret_cast<const int *>(mbar)[RD];
  const float *fold = base + z.off_fold();
  const uint16_t *Ahi = reinterpret_cast<const uint16_t *>(fold);
  const uint16_t *Alo = Ahi + int64_t(HC + HIDDEN) * RD;
  const float *c0 = fold + int64_t(HC + HIDDEN) * RD;     // q0 [HC] then h0 [HIDDEN]
  const uint16_t *w1c_hi =
      reinterpret_cast<const uint16_t *>(shared + align64f(F * HC) + align64f((F + HC) * HIDDEN));
  const uint16_t *w1c_lo = w1c_hi + int64_t(HIDDEN) * HC;
  // blob offsets (packing order of the header)
  const int64_t oWQ = 0, oW1 = HC * F + HC + 2 * (int64_t(HC) * RD + HC);
  const int64_t oW2 = oW1 + int64_t(HIDDEN) * (F + HC) + HIDDEN;
  const float b2 = blob[oW2 + HIDDEN];
  const float alpha = fminf(fmaxf(blob[oW2 + HIDDEN + 1], -5.0f), 5.0f);

  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  float *out = scores + s.slot_off;

  if (t == 0) any = 0;
  __syncthreads();
  if (t < RT) {
    const int j = j0 + t;
    bool c = false;
    if (j < s.N) {
      const int slot = slot_maps[s.slot_off + j];
      c = slot != dead && !(j < s.pi || (j >= s.qs && j < s.qe));
    }
    pos_s[t] = c ? j : -1;
    rule_s[t] = c ? out[j] : 0.f;
    if (c) atomicOr(&any, 1);
  }
  __syncthreads();
  if (!any) return;

  // kbar rows of the tile (and K', V' of the live query positions), split into bf16
  // hi + lo in LDS: eight float4 loads per thread per matrix, all in flight at once
  constexpr int NQ4 = RT * RD / 4 / 256;
  {
    float4 v[NQ4];
#pragma unroll
    for (int q = 0; q < NQ4; ++q) {
      const int e4 = q * 256 + t, r = e4 / (RD / 4), d = (e4 % (RD / 4)) * 4;
      const int j = pos_s[r];
      v[q] = j >= 0 ? *reinterpret_cast<const float4 *>(kbar + int64_t(j) * RD + d) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int q = 0; q < NQ4; ++q) {
      const int e4 = q * 256 + t, r = e4 / (RD / 4), d = (e4 % (RD / 4)) * 4;
      const float x[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) split_bf16(x[k], xs[0][r * XS + d + k], xs[1][r * XS + d + k]);
    }
  }
  const bool on = xattn && nql > 0;
  if (on) {
    float4 kv[NQ4], vv[NQ4];
#pragma unroll
    for (int q = 0; q < NQ4; ++q) {
      const int e4 = q * 256 + t, key = e4 / (RD / 4), d = (e4 % (RD / 4)) * 4;
      const bool live = key < nql;
      kv[q] = live ? *reinterpret_cast<const float4 *>(kp + int64_t(key) * HC + d) : make_float4(0.f, 0.f, 0.f, 0.f);
      vv[q] = live ? *reinterpret_cast<const float4 *>(vp + int64_t(key) * HC + d) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int q = 0; q < NQ4; ++q) {
      const int e4 = q * 256 + t, key = e4 / (RD / 4), d = (e4 % (RD / 4)) * 4;
      const float xk[4] = {kv[q].x, kv[q].y, kv[q].z, kv[q].w};
      const float xv[4] = {vv[q].x, vv[q].y, vv[q].z, vv[q].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        split_bf16(xk[k], kps[0][key * XS + d + k], kps[1][key * XS + d + k]);
        split_bf16(xv[k], vts[0][(d + k) * PS + key], vts[1][(d + k) * PS + key]);
      }
    }
  }
  __syncthreads();

  // ---- 1. [Q ; hidden]: wave w owns output blocks w + 4 i (i = 0, 1: Q; i = 2..5: hidden)
  f32x4 acc[6][4];
#pragma unroll
  for (int i = 0; i < 6; ++i)
#pragma unroll
    for (int tb = 0; tb < 4; ++tb) acc[i][tb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    const int o = (w + 4 * i) * 16 + r16;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 bh = ld8(Ahi + int64_t(o) * RD + ks * 32 + g * 8);
      const bf16x8 bl = ld8(Alo + int64_t(o) * RD + ks * 32 + g * 8);
#pragma unroll
      for (int tb = 0; tb < 4; ++tb) {
        const int r = (tb * 16 + r16) * XS + ks * 32 + g * 8;
        acc[i][tb] = mfma3(ld8(&xs[0][r]), ld8(&xs[1][r]), bh, bl, acc[i][tb]);
      }
    }
  }
  // acc[i][tb][e]: candidate tb*16 + 4g + e, output (w + 4i)*16 + r16; add constant and rule terms
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    const int o = (w + 4 * i) * 16 + r16;
    const float wr = o < HC ? blob[oWQ + int64_t(o) * F + 3 * RD] : blob[oW1 + int64_t(o - HC) * (F + HC) + 3 * RD];
    const float cst = c0[o];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][tb][e] += cst + wr * rule_s[tb * 16 + 4 * g + e];
  }
  __syncthreads();                                   // every wave is done with kbar
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int col = (w + 4 * i) * 16 + r16;
#pragma unroll
    for (int tb = 0; tb < 4; ++tb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        uint16_t h, l;
        split_bf16(acc[i][tb][e], h, l);
        xs[0][(tb * 16 + 4 * g + e) * XS + col] = h;
        xs[1][(tb * 16 + 4 * g + e) * XS + col] = l;
      }
  }
  __syncthreads();

  // ---- 2-3. cross-attention; wave w owns candidates 16w .. 16w+15 (their rows of Q become c)
  if (on) {
    const float sc = 0.17677669529663688f;           // 1/sqrt(32)
    for (int h = 0; h < HC_HEADS; ++h) {
      f32x4 lg[4];
      const int qr = (16 * w + r16) * XS + h * 32 + g * 8;
      const bf16x8 qh = ld8(&xs[0][qr]), ql = ld8(&xs[1][qr]);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int kr = (kb * 16 + r16) * XS + h * 32 + g * 8;
        lg[kb] = mfma3(qh, ql, ld8(&kps[0][kr]), ld8(&kps[1][kr]), f32x4{0.f, 0.f, 0.f, 0.f});
      }
      // lg[kb][e]: candidate 16w + 4g + e, key kb*16 + r16
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float m = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          lg[kb][e] = (kb * 16 + r16 < nql) ? lg[kb][e] * sc : -INFINITY;
          m = fmaxf(m, lg[kb][e]);
        }
        m = fmaxf(m, __shfl_xor(m, 1, WAVE));
        m = fmaxf(m, __shfl_xor(m, 2, WAVE));
        m = fmaxf(m, __shfl_xor(m, 4, WAVE));
        m = fmaxf(m, __shfl_xor(m, 8, WAVE));
        float sum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          lg[kb][e] = expf(lg[kb][e] - m);
          sum += lg[kb][e];
        }
        sum += __shfl_xor(sum, 1, WAVE);
        sum += __shfl_xor(sum, 2, WAVE);
        sum += __shfl_xor(sum, 4, WAVE);
        sum += __shfl_xor(sum, 8, WAVE);
        const float inv = 1.0f / sum;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          uint16_t ph, pl;
          split_bf16(lg[kb][e] * inv, ph, pl);
          ps[0][(16 * w + 4 * g + e) * PS + kb * 16 + r16] = ph;
          ps[1][(16 * w + 4 * g + e) * PS + kb * 16 + r16] = pl;
        }
      }
      // c_h = P . V'_h (the weights were written by this wave; its LDS ops run in order)
      f32x4 cc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int pr = (16 * w + r16) * PS + ks * 32 + g * 8;
        const bf16x8 ph = ld8(&ps[0][pr]), pl = ld8(&ps[1][pr]);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const int vr = (h * 32 + nb * 16 + r16) * PS + ks * 32 + g * 8;
          cc[nb] = mfma3(ph, pl, ld8(&vts[0][vr]), ld8(&vts[1][vr]), cc[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint16_t ch, cl;
          split_bf16(cc[nb][e], ch, cl);
          const int idx = (16 * w + 4 * g + e) * XS + h * 32 + nb * 16 + r16;
          xs[0][idx] = ch;
          xs[1][idx] = cl;
        }
    }
    __syncthreads();
    // ---- 4. hidden += c . W_1^c^T for this wave's hidden blocks
#pragma unroll
    for (int i = 2; i < 6; ++i) {
      const int oh = (w + 4 * i - 8) * 16 + r16;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 bh = ld8(w1c_hi + int64_t(oh) * HC + ks * 32 + g * 8);
        const bf16x8 bl = ld8(w1c_lo + int64_t(oh) * HC + ks * 32 + g * 8);
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) {
          const int r = (tb * 16 + r16) * XS + ks * 32 + g * 8;
          acc[i][tb] = mfma3(ld8(&xs[0][r]), ld8(&xs[1][r]), bh, bl, acc[i][tb]);
        }
      }
    }
  }

  // ---- y = w_2 . GELU(hidden) + b_2, reduced over the 256 hidden units
  float ys[4][4];
#pragma unroll
  for (int tb = 0; tb < 4; ++tb)
#pragma unroll
    for (int e = 0; e < 4; ++e) ys[tb][e] = 0.f;
#pragma unroll
  for (int i = 2; i < 6; ++i) {
    const int oh = (w + 4 * i - 8) * 16 + r16;
    const float w2 = blob[oW2 + oh];
#pragma unroll
    for (int tb = 0; tb < 4; ++tb)
#pragma unroll
      for (int e = 0; e < 4; ++e) ys[tb][e] = fmaf(gelu_exact(acc[i][tb][e]), w2, ys[tb][e]);
  }
#pragma unroll
  for (int tb = 0; tb < 4; ++tb)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = ys[tb][e];
      v += __shfl_xor(v, 1, WAVE);
      v += __shfl_xor(v, 2, WAVE);
      v += __shfl_xor(v, 4, WAVE);
      v += __shfl_xor(v, 8, WAVE);
      if (r16 == 0) red[w][tb * 16 + 4 * g + e] = v;
    }
  __syncthreads();
  if (t < RT && pos_s[t] >= 0) {
    const float y = ((red[0][t] + red[1][t]) + (red[2][t] + red[3][t])) + b2;
    out[pos_s[t]] = rule_s[t] + alpha * y;
  }
}

hipError_t launch_residual_mfma(const ScoreArgs &a, hipStream_t st) {
  const ikv_pool &p = a.pool;
  {
    KTimer kt_("k_residual_mfma", st);
    k_residual_mfma<<<dim3(unsigned(cdiv(a.maxN, RT)), a.B), 256, 0, st>>>(
        a.sess_dev, a.slot_maps, p.dead_slot, a.scores, a.ws, a.ws_shared, a.residual, p.L, p.Hkv,
        (a.flags & IKV_NO_XATTN) == 0);
  }
  return hipGetLastError();
}

}  // namespace ikv
