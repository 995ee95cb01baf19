// Residual head of Eq. 4 (features Eq. 5, cross-attention Eq. 6) on the matrix cores,
// for D = 128 and at most 64 live query positions per session.
//
// With mbar folded into the first-layer weights (res_fold_wg, which runs in the
// row-statistics launch), the head of one candidate is a chain of small products on
// v_mfma_f32_16x16x32_bf16. Each wave owns 16 candidates and keeps its activations in
// registers: the products run transposed (weights as the A operand, candidates as the
// columns), so that the accumulator of one product is, lane for lane, the B operand
// of the next, up to the order of the contraction index inside each 32-wide block
// (perm32), which the pre-arranged K', V' and W_1^c fragments follow:
//   1. Q^T = A_Q kbar^T + q0 + w_Q^r rule                      (128 x 16, K = 128)
//   2. logits_h^T = K'_h Q_h^T / sqrt(32)                      (per head, 64 x 16, K = 32)
//   3. c_h^T = V'_h^T softmax(logits_h)^T                      (per head, 32 x 16, K = 64)
//   4. hidden^T = A_1 kbar^T + W_1^c c^T + h0 + w_1^r rule     (256 x 16, K = 128 + 128)
// then y = w_2 . GELU(hidden) + b_2 and s = rule + clip(alpha, -5, 5) y. Every operand
// is split into bf16 hi + lo and each product runs as hi.hi + hi.lo + lo.hi with
// float32 accumulation (relative error about 2^-17 per product).
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int RD = 128;          // head dimension of this path
constexpr int RW = 16;           // candidates per wave
constexpr int RWAVES = 8;        // waves per workgroup (one workgroup per CU)
constexpr int RT = RWAVES * RW;  // candidates per workgroup
constexpr int RKI = 16 / RWAVES; // 1-KB loads per wave per weight stage
static_assert(HC == 128 && HC_HEADS == 4 && HIDDEN == 256, "fragment layout of this path");

__device__ __forceinline__ bf16x8 ld8(const uint16_t *p) { return *reinterpret_cast<const bf16x8 *>(p); }

// v = hi + lo in bf16, both rounded to nearest even (the conversion instruction of gfx950)
__device__ __forceinline__ void split8(const float (&v)[8], bf16x8 &h, bf16x8 &l) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    h[e] = __bf16(v[e]);
    l[e] = __bf16(v[e] - float(h[e]));
  }
}

__device__ __forceinline__ f32x4 mfma3(const bf16x8 &ah, const bf16x8 &al, const bf16x8 &bh, const bf16x8 &bl,
                                       f32x4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
  return acc;
}

// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, formula 7.1.26
// (absolute error at most 1.5e-7), extended to negative arguments by oddness.
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  const float p = t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f),
                           0.254829592f);
  const float r = 1.0f - p * __builtin_amdgcn_exp2f(-ax * ax * 1.4426950408889634f);
  return copysignf(r, x);
}

__device__ __forceinline__ float gelu_as(float x) { return 0.5f * x * (1.0f + erf_as(x * 0.70710678118654752f)); }

// The weights stream once per workgroup through a 9-stage LDS ring of 16 KB stages
// (direct global->LDS loads, eight stages in flight, waits placed by hand), shared by
// the eight waves:
//   stages 0..3    rows 32 s .. + 31 of A_Q, hi then lo;
//   stages 4..7    K' then V' fragments of head s - 4;
//   stages 8..23   rows 16 ob .. + 15 of A_1 (hi, lo) and of W_1^c (hi, lo), ob = s - 8.
// Weight rows are 256 B with 16-byte chunk c of row r at slot c ^ (r & 15), so the 16
// rows of a fragment read hit distinct banks.
constexpr int RS_STAGES = 9;
constexpr int RS_STAGE = 8192;                   // bf16 per stage (16 KB)
constexpr int RS_NSTAGE = 24;

__device__ __forceinline__ void dma16r(const void *g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds_base), "v"(g)
               : "memory", "m0");
}

// s_waitcnt vmcnt(n) for a wave-uniform even n in 0..14
__device__ __forceinline__ void rs_wait(int n) {
  switch (n) {
    case 2: asm volatile("s_waitcnt vmcnt(2)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(6)" ::: "memory"); break;
    case 8: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
    case 10: asm volatile("s_waitcnt vmcnt(10)" ::: "memory"); break;
    case 12: asm volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
    case 14: asm volatile("s_waitcnt vmcnt(14)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
}

__global__ void __launch_bounds__(64 * RWAVES) __attribute__((amdgpu_waves_per_eu(2)))
k_residual_mfma(const ikv_session *__restrict__ sess, const int32_t *__restrict__ slot_maps, int dead,
                float *__restrict__ scores, const float *__restrict__ ws, const float *__restrict__ shared,
                const float *__restrict__ blob, int L, int Hkv, bool xattn, int CH) {
  __shared__ __align__(1024) uint16_t ring[RS_STAGES * RS_STAGE];
  __shared__ __align__(16) float cst[2 * (HC + HIDDEN) + HIDDEN];   // q0 | h0, rule column, w_2
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int g = lane >> 4, i = lane & 15;
  // list tile k of chunk c takes entries [c CH + 128 k, + 128) of the candidate list; the
  // grid runs tile-index-major (block x = k * chunks + c), which spreads the tiles of
  // sparse chunks over the XCDs
  const int per = CH / RT, nch = int(gridDim.x) / per;
  const int lc = int(blockIdx.x) % nch, lk = int(blockIdx.x) / nch;
  if (int64_t(lc) * CH >= s.N) return;
  const int units = L * Hkv;
  constexpr int64_t F = 3 * RD + 1;
  const ScoreSizes z = score_sizes(s, L, units, RD, true, true);
  const float *base = ws + score_offset(sess, b, L, units, RD, true, true);
  const float *kbar = base + z.off_kbar();
  const float *mbar = base + z.off_misc() + int64_t(MBAR_PARTS) * RD;
  const int nql = reinterpret_cast<const int *>(mbar)[RD];
  const float *fold = base + z.off_fold();
  const uint16_t *Ahi = reinterpret_cast<const uint16_t *>(fold);
  const uint16_t *Alo = Ahi + int64_t(HC + HIDDEN) * RD;
  const float *c0 = fold + int64_t(HC + HIDDEN) * RD;    // q0 [HC], h0 [HIDDEN], then the rule column
  const uint16_t *kf = reinterpret_cast<const uint16_t *>(base + z.off_kvf());
  const uint16_t *vf = kf + KVF_BF16 / 2;
  const uint16_t *w1c_hi =
      reinterpret_cast<const uint16_t *>(shared + align64f(F * HC) + align64f((F + HC) * HIDDEN));
  const uint16_t *w1c_lo = w1c_hi + int64_t(HIDDEN) * HC;
  const int64_t oW2 = HC * F + HC + 2 * (int64_t(HC) * RD + HC) + int64_t(HIDDEN) * (F + HC) + HIDDEN;
  const float b2 = blob[oW2 + HIDDEN];
  const float alpha = fminf(fmaxf(blob[oW2 + HIDDEN + 1], -5.0f), 5.0f);
  float *out = scores + s.slot_off;

  // lane (g, i) of wave w works for list entry 16 w + i of the tile (a candidate)
  const int32_t *lst = reinterpret_cast<const int32_t *>(base + z.off_clist()) + lc * CH + lk * RT;
  const int cnt = reinterpret_cast<const int32_t *>(base + z.off_ccount(s.N))[lc];
  const int ne = min(RT, cnt - lk * RT);
  if (ne <= 0) return;
  const bool ident = cnt == min(CH, s.N - lc * CH);   // every position a candidate: its own list
  const int e = RW * w + i;
  const bool cand = e < ne;
  const int ec = cand ? e : ne - 1;
  const int j = ident ? lc * CH + lk * RT + ec : lst[ec], jc = j;
  if (!__syncthreads_or(cand)) return;
  const float rule = out[jc];
  for (int k = t; k < 2 * (HC + HIDDEN); k += 64 * RWAVES) cst[k] = c0[k];
  for (int k = t; k < HIDDEN; k += 64 * RWAVES) cst[2 * (HC + HIDDEN) + k] = blob[oW2 + k];

  // kbar^T as the B operand: lane (g, i) holds channels 32 ks + 8 g .. + 7 of its candidate
  bf16x8 xh[4], xl[4];
  {
    float4 v[8];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float *src = kbar + int64_t(jc) * RD + 32 * ks + 8 * g;
      v[2 * ks] = *reinterpret_cast<const float4 *>(src);
      v[2 * ks + 1] = *reinterpret_cast<const float4 *>(src + 4);
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const float x[8] = {v[2 * ks].x,     v[2 * ks].y,     v[2 * ks].z,     v[2 * ks].w,
                          v[2 * ks + 1].x, v[2 * ks + 1].y, v[2 * ks + 1].z, v[2 * ks + 1].w};
      split8(x, xh[ks], xl[ks]);
    }
  }
  // every compiler-issued load of the set-up is complete before the first weight load
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // stage st, wave w, instruction k fills 1 KB: n = RKI w + k
  const uint32_t ring0 = uint32_t(reinterpret_cast<uintptr_t>(ring));
  auto issue = [&](int st) {
    if (st >= RS_NSTAGE) return;
    const uint32_t dst = ring0 + uint32_t((st % RS_STAGES) * RS_STAGE * 2);
#pragma unroll
    for (int k = 0; k < RKI; ++k) {
      const int n = RKI * w + k;
      const uint16_t *src;
      if (st < 4) {                                // 32 rows of A_Q: hi (n < 8), lo
        const int r = 4 * (n & 7) + (lane >> 4);
        src = (n < 8 ? Ahi : Alo) + int64_t(32 * st + r) * RD + (((lane & 15) ^ (r & 15)) * 8);
      } else if (st < 8) {                         // fragments of head st - 4: K' (n < 8), V'
        src = (n < 8 ? kf : vf) + (st - 4) * 4096 + (n & 7) * 512 + lane * 8;
      } else {                                     // 16 rows of A_1 hi, lo, W_1^c hi, lo
        const int part = n >> 2, r = 4 * (n & 3) + (lane >> 4);
        const uint16_t *m = part == 0 ? Ahi : part == 1 ? Alo : part == 2 ? w1c_hi : w1c_lo;
        const int row = (part < 2 ? HC : 0) + 16 * (st - 8) + r;
        src = m + int64_t(row) * RD + (((lane & 15) ^ (r & 15)) * 8);
      }
      dma16r(src, __builtin_amdgcn_readfirstlane(dst + uint32_t(n * 1024)));
    }
  };
  // top of stage st: its loads are done once at most those of the later stages already
  // issued (RKI each) are outstanding; the barrier also frees the buffer of stage st - 1
  auto advance = [&](int st) {
    rs_wait(RKI * min(RS_STAGES - 2, RS_NSTAGE - 1 - st));
    __syncthreads();
    issue(st + RS_STAGES - 1);
    return ring + (st % RS_STAGES) * RS_STAGE;
  };
  // 16 weight rows at `rows` (hi) and `rows + lo_off` (lo) against kbar^T
  auto rows_x_kbar = [&](const uint16_t *rows, int lo_off) {
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int o = i * RD + (((4 * ks + g) ^ i) * 8);
      acc = mfma3(ld8(rows + o), ld8(rows + lo_off + o), xh[ks], xl[ks], acc);
    }
    return acc;
  };
  // constant and rule terms of output rows 16 ob + 4 g + e
  auto add_terms = [&](f32x4 &acc, int ob) {
    const float4 cv = *reinterpret_cast<const float4 *>(cst + 16 * ob + 4 * g);
    const float4 rv = *reinterpret_cast<const float4 *>(cst + HC + HIDDEN + 16 * ob + 4 * g);
    acc[0] += fmaf(rv.x, rule, cv.x);
    acc[1] += fmaf(rv.y, rule, cv.y);
    acc[2] += fmaf(rv.z, rule, cv.z);
    acc[3] += fmaf(rv.w, rule, cv.w);
  };

  for (int k = 0; k < RS_STAGES - 1; ++k) issue(k);

  // ---- Q^T: lane (g, i) gets channels 16 ob + 4 g + e of its candidate
  f32x4 q[8];
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const uint16_t *sp = advance(st);
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      q[2 * st + blk] = rows_x_kbar(sp + blk * 16 * RD, 32 * RD);
      add_terms(q[2 * st + blk], 2 * st + blk);
    }
  }

  // ---- cross-attention: c^T fragments per head (zero without live query positions)
  bf16x8 ch[HC_HEADS], cl[HC_HEADS];
  const bool on = xattn && nql > 0;
  const float sc = 1.4426950408889634f * 0.17677669529663688f;   // log2(e) / sqrt(32)
#pragma unroll
  for (int h = 0; h < HC_HEADS; ++h) {
    const uint16_t *sp = advance(4 + h);
#pragma unroll
    for (int e = 0; e < 8; ++e) ch[h][e] = cl[h][e] = __bf16(0.0f);
    if (!on) continue;
    // Q_h^T: channels 32 h + perm32(g, e) of the candidate, from output blocks 2h and 2h + 1
    bf16x8 qh, ql;
    {
      const float x[8] = {q[2 * h][0], q[2 * h][1], q[2 * h][2], q[2 * h][3],
                          q[2 * h + 1][0], q[2 * h + 1][1], q[2 * h + 1][2], q[2 * h + 1][3]};
      split8(x, qh, ql);
    }
    f32x4 lg[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const uint16_t *kp = sp + (kb * 2) * 512 + lane * 8;
      lg[kb] = mfma3(ld8(kp), ld8(kp + 512), qh, ql, f32x4{0.f, 0.f, 0.f, 0.f});
    }
    // lg[kb][e]: key 16 kb + 4 g + e; softmax over the live keys of candidate i
    float m = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lg[kb][e] = (16 * kb + 4 * g + e < nql) ? lg[kb][e] * sc : -INFINITY;
        m = fmaxf(m, lg[kb][e]);
      }
    m = fmaxf(m, __shfl_xor(m, 16, WAVE));
    m = fmaxf(m, __shfl_xor(m, 32, WAVE));
    float sum = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lg[kb][e] = __builtin_amdgcn_exp2f(lg[kb][e] - m);
        sum += lg[kb][e];
      }
    sum += __shfl_xor(sum, 16, WAVE);
    sum += __shfl_xor(sum, 32, WAVE);
    const float inv = 1.0f / sum;
    // P^T for key step ks: keys 32 ks + perm32(g, e) are lg[2 ks] and lg[2 ks + 1]
    f32x4 cc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 ph, pl;
      const float x[8] = {lg[2 * ks][0] * inv,     lg[2 * ks][1] * inv,     lg[2 * ks][2] * inv,
                          lg[2 * ks][3] * inv,     lg[2 * ks + 1][0] * inv, lg[2 * ks + 1][1] * inv,
                          lg[2 * ks + 1][2] * inv, lg[2 * ks + 1][3] * inv};
      split8(x, ph, pl);
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const uint16_t *vp = sp + 4096 + ((nb * 2 + ks) * 2) * 512 + lane * 8;
        cc[nb] = mfma3(ld8(vp), ld8(vp + 512), ph, pl, cc[nb]);
      }
    }
    // cc[nb][e]: channel 32 h + 16 nb + 4 g + e, i.e. k index perm32 of c^T for the last layer
    const float x[8] = {cc[0][0], cc[0][1], cc[0][2], cc[0][3], cc[1][0], cc[1][1], cc[1][2], cc[1][3]};
    split8(x, ch[h], cl[h]);
  }

  // ---- hidden^T, 16 units per stage, then w_2 . GELU summed over this lane's units
  float ys = 0.f;
  for (int ob = 0; ob < HIDDEN / 16; ++ob) {
    const uint16_t *sp = advance(8 + ob);
    f32x4 acc = rows_x_kbar(sp, 16 * RD);
    if (on) {
#pragma unroll
      for (int h = 0; h < HC_HEADS; ++h) {
        const int o = i * RD + (((4 * h + g) ^ i) * 8);
        acc = mfma3(ld8(sp + 32 * RD + o), ld8(sp + 48 * RD + o), ch[h], cl[h], acc);
      }
    }
    add_terms(acc, HC / 16 + ob);
    const float4 w2v = *reinterpret_cast<const float4 *>(cst + 2 * (HC + HIDDEN) + 16 * ob + 4 * g);
    ys = fmaf(gelu_as(acc[0]), w2v.x, ys);
    ys = fmaf(gelu_as(acc[1]), w2v.y, ys);
    ys = fmaf(gelu_as(acc[2]), w2v.z, ys);
    ys = fmaf(gelu_as(acc[3]), w2v.w, ys);
  }
  ys += __shfl_xor(ys, 16, WAVE);
  ys += __shfl_xor(ys, 32, WAVE);
  if (g == 0 && cand) out[j] = rule + alpha * (ys + b2);
}

hipError_t launch_residual_mfma(const ScoreArgs &a, hipStream_t st) {
  const ikv_pool &p = a.pool;
  {
    KTimer kt_("k_residual_mfma", st);
    const int lch = stats_chunk(a.maxN, std::max(1, p.L * p.Hkv / 2));   // the candidate lists' chunk
    k_residual_mfma<<<dim3(unsigned(cdiv(a.maxN, lch) * (lch / RT)), a.B), 64 * RWAVES, 0, st>>>(
        a.sess_dev, a.slot_maps, p.dead_slot, a.scores, a.ws, a.ws_shared, a.residual, p.L, p.Hkv,
        (a.flags & IKV_NO_XATTN) == 0, lch);
  }
  return hipGetLastError();
}

}  // namespace ikv
