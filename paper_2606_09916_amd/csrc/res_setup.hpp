// Per-session set-up of the residual head (Eqs. 4-6): mbar, the live query positions,
// the first-layer weights with mbar folded in, and K', V' of the live query rows.
// Shared by the stand-alone residual kernels and by the workgroups that the
// row-statistics launch adds for them.
#pragma once
#include "ikv_internal.hpp"

namespace ikv {

// Offsets (floats) of the parameter blocks in the packed blob.
struct ResLayout {
  int64_t WQ, bQ, WK, bK, WV, bV, W1, b1, w2, b2, alpha, total;
  __host__ __device__ explicit ResLayout(int D) {
    const int64_t F = 3 * D + 1;
    WQ = 0;
    bQ = WQ + HC * F;
    WK = bQ + HC;
    bK = WK + int64_t(HC) * D;
    WV = bK + HC;
    bV = WV + int64_t(HC) * D;
    W1 = bV + HC;
    b1 = W1 + int64_t(HIDDEN) * (F + HC);
    w2 = b1 + HIDDEN;
    b2 = w2 + HIDDEN;
    alpha = b2 + 1;
    total = alpha + 1;
  }
};

// Sum of the np partial rows parts [np][D] per channel, in a fixed order: NT / D
// threads per channel each add every (NT / D)-th row in order, and their sums are
// added in thread order. Returns channel t's sum in thread t < D. Every thread of the
// workgroup calls it (one barrier); threads past NT only meet the barrier.
template <int D, int NT>
__device__ __forceinline__ float column_sum(const float *__restrict__ parts, int np) {
  constexpr int TPC = NT / D;
  constexpr int U = 24;                            // partial rows in flight per thread
  __shared__ float red[TPC][D];
  const int t = threadIdx.x, c = t % D, grp = t / D;
  if (t < NT) {
    float a = 0.f;
    for (int p0 = grp; p0 < np; p0 += U * TPC) {
      float v[U];
#pragma unroll
      for (int q = 0; q < U; ++q) v[q] = parts[int64_t(min(p0 + q * TPC, np - 1)) * D + c];
#pragma unroll
      for (int q = 0; q < U; ++q)
        if (p0 + q * TPC < np) a += v[q];
    }
    red[grp][c] = a;
  }
  __syncthreads();
  float tot = 0.f;
  if (t < D)
#pragma unroll
    for (int k = 0; k < TPC; ++k) tot += red[k][t];
  return tot;
}

// mbar of session s in thread t < D: the partial column sums (MBAR_PARTS row ranges, or
// with `pairs` one per head pair) added by column_sum over NT threads, over the number
// of memory rows.
template <int D, int NT>
__device__ __forceinline__ float mbar_channel(const ikv_session &s, const float *base, const ScoreSizes &z,
                                              int units, bool pairs) {
  const float *parts = pairs ? base + z.off_mbp() : base + z.off_misc();
  const float tot = column_sum<D, NT>(parts, pairs ? units / 2 : MBAR_PARTS);
  return tot / float(int64_t(units) * s.R);
}

// Session b: mbar and the live query positions in order, to the workspace. Needs at
// least 256 threads; every thread of the workgroup must call it.
template <int D>
__device__ __forceinline__ void res_setup_body(const ikv_session *__restrict__ sess, int b,
                                               const int32_t *__restrict__ slot_maps,
                                               const int32_t *__restrict__ qpos, int dead, float *__restrict__ ws,
                                               int L, int Hkv, bool mfma, bool pairs) {
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const ScoreSizes z = score_sizes(s, L, units, D, true, mfma);
  float *base = ws + score_offset(sess, b, L, units, D, true, mfma);
  float *mbar = base + z.off_misc() + int64_t(MBAR_PARTS) * D;
  int *qlist = reinterpret_cast<int *>(base + z.off_qlist());
  const int t = threadIdx.x;
  const float mb = mbar_channel<D, 256>(s, base, z, units, pairs);
  if (t < D) mbar[t] = mb;
  if (t < WAVE) {   // live query positions in order: one wave, ranked by ballot
    int n = 0;
    const int32_t *S = slot_maps + s.slot_off;
    const int32_t *qp = qpos + s.qpos_off;
    for (int i0 = 0; i0 < s.nq; i0 += WAVE) {
      const int i = i0 + t;
      int j = -1;
      if (i < s.nq) j = qp[i];
      const bool ok = j >= 0 && j < s.N && S[j] != dead;
      const uint64_t bal = __ballot(ok);
      if (ok) qlist[n + __popcll(bal & ((uint64_t(1) << t) - 1))] = j;
      n += __popcll(bal);
    }
    if (t == 0) reinterpret_cast<int *>(mbar)[D] = n;
  }
}

// Folded first layer of one session (exact in real arithmetic):
//   W_Q phi + b_Q  = (W_Q^k + W_Q^km diag(mbar)) kbar + (W_Q^m mbar + b_Q) + w_Q^r rule
//   W_1 [phi; c] + b_1 = (W_1^k + W_1^km diag(mbar)) kbar + (W_1^m mbar + b_1) + w_1^r rule + W_1^c c
// Rows 0..HC-1 of the folded matrix are the W_Q part, rows HC.. the W_1 part; stored
// as bf16 hi [HC+HIDDEN][D] then lo, then q0 [HC] and h0 [HIDDEN] in float32, then
// the rule column w_Q^r [HC] and w_1^r [HIDDEN]. The items of the fold, one per
// thread: the folded matrix (one element each), q0 | h0 (Q0_PARTS adjacent threads per
// row), the rule column, and last (session 0 only) the cross-attention columns of W_1,
// shared by every session. A session at or under its budget has no mbar and takes only
// the shared items.
constexpr int Q0_PARTS = 4;
template <int D> constexpr int64_t fold_own_items() {
  return int64_t(HC + HIDDEN) * D + (Q0_PARTS + 1) * (HC + HIDDEN);
}
template <int D> constexpr int64_t fold_items() { return fold_own_items<D>() + int64_t(HIDDEN) * HC; }

// Workgroup fw of the fold of session b: item fw * 512 + t in thread t (the launch has
// one thread per item). The operands that do not depend on mbar are loaded first;
// mbar is then recomputed from its partial sums over all 512 threads, so that the fold
// needs nothing from the set-up workgroup of the same launch. Needs 512 threads; every
// thread calls it.
template <int D>
__device__ __forceinline__ void res_fold_wg(int fw, const ikv_session *__restrict__ sess, int b,
                                            const float *__restrict__ blob, float *__restrict__ ws,
                                            float *__restrict__ shared, int L, int Hkv, bool pairs) {
  constexpr int RB = D / Q0_PARTS;                 // q0 row elements per thread
  static_assert((int64_t(HC + HIDDEN) * D) % WAVE == 0 && (Q0_PARTS * (HC + HIDDEN)) % WAVE == 0,
                "the q0 items fill whole wavefronts");
  const ikv_session s = sess[b];
  const bool skipped = s.N <= s.C;
  const ResLayout lay(D);
  const int64_t F = 3 * D + 1;
  const int64_t nw = int64_t(HC + HIDDEN) * D, nq0 = nw + Q0_PARTS * (HC + HIDDEN);
  const int64_t own = fold_own_items<D>();         // the session's own items; the shared ones follow
  const int64_t i0 = int64_t(fw) * blockDim.x, i = i0 + threadIdx.x;
  if ((skipped || i0 >= own) && b != 0) return;
  if (skipped && i0 + blockDim.x <= own) return;
  const int units = L * Hkv;
  const ScoreSizes z = score_sizes(s, L, units, D, true, true);
  float *base = ws + score_offset(sess, b, L, units, D, true, true);
  float *fold = base + z.off_fold();
  auto row_of = [&](int64_t o) __attribute__((always_inline)) {
    return o < HC ? blob + lay.WQ + o * F : blob + lay.W1 + (o - HC) * (F + HC);
  };
  // operands that do not need mbar
  float x0 = 0.f, x1 = 0.f, rv[RB];
  if (i < nw) {
    const int64_t o = i / D, d = i - o * D;
    x0 = row_of(o)[d];
    x1 = row_of(o)[2 * D + d];
  } else if (i < nq0) {
    const int64_t o = (i - nw) / Q0_PARTS;
    const int part = int(i - nw) % Q0_PARTS;
    if (part == 0) x0 = o < HC ? blob[lay.bQ + o] : blob[lay.b1 + (o - HC)];
#pragma unroll
    for (int d = 0; d < RB; ++d) rv[d] = row_of(o)[D + RB * part + d];
  } else if (i < own) {
    x0 = row_of(i - nq0)[3 * D];
  } else if (b == 0 && i < fold_items<D>()) {
    const int64_t k = i - own, oc = k / HC, c = k - oc * HC;
    x0 = blob[lay.W1 + oc * (F + HC) + F + c];
  }
  __shared__ float mb[D];
  if (!skipped) {
    const float m = mbar_channel<D, 512>(s, base, z, units, pairs);
    if (threadIdx.x < D) mb[threadIdx.x] = m;
    __syncthreads();
  }
  uint16_t *hi = reinterpret_cast<uint16_t *>(fold);
  uint16_t *lo = hi + nw;
  float *q0 = fold + nw;
  if (i < nw) {
    if (skipped) return;
    const float v = fmaf(x1, mb[i % D], x0);
    const uint16_t h = float_to_bf16_bits(v);
    hi[i] = h;
    lo[i] = float_to_bf16_bits(v - bf16_bits_to_float(h));
  } else if (i < nq0) {
    // every lane of these wavefronts holds a q0 part (the region is whole workgroups)
    if (skipped) return;
    const int part = int(i - nw) % Q0_PARTS;
    float a = 0.f;
#pragma unroll
    for (int d = 0; d < RB; ++d) a = fmaf(rv[d], mb[RB * part + d], a);
    a += __shfl_xor(a, 1, WAVE);                   // parts (0 + 1) and (2 + 3), then their sum
    a += __shfl_xor(a, 2, WAVE);
    if (part == 0) q0[(i - nw) / Q0_PARTS] = x0 + a;
  } else if (i < own) {                             // the rule column
    if (skipped) return;
    q0[HC + HIDDEN + (i - nq0)] = x0;
  } else if (b == 0 && i < fold_items<D>()) {
    // the cross-attention columns of W_1 as bf16 hi + lo [HIDDEN][HC], each 32-wide
    // head block in the MFMA k order of perm32
    uint16_t *w1c = reinterpret_cast<uint16_t *>(shared + align64f(F * HC) + align64f((F + HC) * HIDDEN));
    const int64_t k = i - own, nc = int64_t(HIDDEN) * HC;
    const int64_t oc = k / HC, c = k - oc * HC;
    const uint16_t h = float_to_bf16_bits(x0);
    const int64_t at = oc * HC + (c & ~int64_t(31)) + perm32_inv(int(c & 31));
    w1c[at] = h;
    w1c[nc + at] = float_to_bf16_bits(x0 - bf16_bits_to_float(h));
  }
}

// K' and V' of live query row `key` (value v of output o: K' for o < HC, V' after) as
// bf16 hi + lo MFMA fragments, zeros past the live rows (`live` false):
//   K' [head][key block kb][hi|lo][lane 16 g + i][8]: key 16 kb + i, channels
//      32 head + perm32(g, e) (the A operand of the logits block);
//   V' [head][channel block nb][key step ks][hi|lo][lane 16 g + i][8]: channel
//      32 head + 16 nb + i, keys 32 ks + perm32(g, e) (the A operand of the context).
__device__ __forceinline__ void res_kv_frag_store(uint16_t *__restrict__ kf, uint16_t *__restrict__ vf, int key, int o,
                                                  float v) {
  const bool isv = o >= HC;
  const int oc = o & (HC - 1);
  const int head = oc >> 5, c = oc & 31;
  const uint16_t hi = float_to_bf16_bits(v), lo = float_to_bf16_bits(v - bf16_bits_to_float(hi));
  if (!isv) {
    const int k = perm32_inv(c), kb = key >> 4, lane = 16 * (k >> 3) + (key & 15);
    const int64_t at = int64_t((head * 4 + kb) * 2) * 512 + lane * 8 + (k & 7);
    kf[at] = hi;
    kf[at + 512] = lo;
  } else {
    const int nb = c >> 4, ks = key >> 5, k = perm32_inv(key & 31), lane = 16 * (k >> 3) + (c & 15);
    const int64_t at = int64_t(((head * 2 + nb) * 2 + ks) * 2) * 512 + lane * 8 + (k & 7);
    vf[at] = hi;
    vf[at + 512] = lo;
  }
}

// Row `key` (< RES_KEYS) of K' = W_K kq + b_K and V' = W_V kq + b_V for session b (D =
// 128, bf16 keys), written as floats and as fragments (res_kv_frag_store). kq, the mean
// key row at the key-th live query position, is summed here from the keys themselves
// (Eq. 5's mean over layers and KV heads), so that it needs nothing from the second
// pass: 32 groups of 16 threads each add the rows of every 32nd unit in order, and the
// groups' sums are added in group order. Thread t computes half (t / 256) of output
// t % 256; its weights are loaded before the keys arrive. Needs 512 threads; every
// thread calls it.
template <int D>
__device__ __forceinline__ void res_kv_keys_wg(int key, const ikv_session *__restrict__ sess, int b,
                                               const uint16_t *__restrict__ kpool, int64_t num_slots, int L,
                                               int Hkv, const int32_t *__restrict__ slot_maps,
                                               const int32_t *__restrict__ qpos, int dead,
                                               const float *__restrict__ blob, float *__restrict__ ws) {
  static_assert(D == 128, "sixteen 16-byte pieces per key row");
  constexpr int NG = 32;                           // unit groups
  constexpr int DH = D / 2;                        // weights per thread
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const ResLayout lay(D);
  const ScoreSizes z = score_sizes(s, L, units, D, true, true);
  float *base = ws + score_offset(sess, b, L, units, D, true, true);
  const int t = threadIdx.x;
  __shared__ int sel[2];                           // live count, the slot of the key-th live position
  __shared__ float red[NG][D + 4];
  __shared__ float kq[D];
  __shared__ float half1[2 * HC];
  if (t < WAVE) {   // the key-th live query position, by the ballot ranking of res_setup_body
    int n = 0, slot = -1;
    const int32_t *S = slot_maps + s.slot_off;
    const int32_t *qp = qpos + s.qpos_off;
    for (int i0 = 0; i0 < s.nq; i0 += WAVE) {
      const int i = i0 + t;
      int j = -1, sj = dead;
      if (i < s.nq) j = qp[i];
      if (j >= 0 && j < s.N) sj = S[j];
      const bool ok = j >= 0 && j < s.N && sj != dead;
      const uint64_t bal = __ballot(ok);
      if (ok && n + __popcll(bal & ((uint64_t(1) << t) - 1)) == key) slot = sj;
      n += __popcll(bal);
    }
    const uint64_t hit = __ballot(slot >= 0);
    if (t == 0) sel[0] = n;
    if (hit && t == __ffsll(static_cast<long long>(hit)) - 1) sel[1] = slot;
  }
  // this thread's half row of W_K (outputs 0..HC-1) or W_V (HC..), independent of kq
  const int o = t & (2 * HC - 1), hf = t >> 8;
  const bool isv = o >= HC;
  float wv[DH];
  const float bias = hf == 0 ? blob[(isv ? lay.bV : lay.bK) + (o & (HC - 1))] : 0.f;
  {
    const float *W = blob + (isv ? lay.WV : lay.WK) + int64_t(o & (HC - 1)) * D + DH * hf;
#pragma unroll
    for (int d = 0; d < DH; ++d) wv[d] = W[d];
  }
  __syncthreads();
  const bool live = key < sel[0];
  if (live) {
    const int64_t slot = sel[1];
    const int c = t & 15, grp = t >> 4;
    float a[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] = 0.f;
    constexpr int U = 9;                           // rows in flight per thread
    for (int u0 = grp; u0 < units; u0 += U * NG) {
      uint4 r[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const int u = min(u0 + q * NG, units - 1), l = u / Hkv, h = u - l * Hkv;
        r[q] = *reinterpret_cast<const uint4 *>(kpool + ((int64_t(l) * num_slots + slot) * Hkv + h) * D + 8 * c);
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
        if (u0 + q * NG >= units) break;
        const uint32_t w4[4] = {r[q].x, r[q].y, r[q].z, r[q].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {              // bf16 -> float is exact: the high half of the word
          a[2 * e] += __uint_as_float(w4[e] << 16);
          a[2 * e + 1] += __uint_as_float(w4[e] & 0xffff0000u);
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) red[grp][8 * c + e] = a[e];
  }
  __syncthreads();
  if (live && t < D) {
    float tot = 0.f;
#pragma unroll 8
    for (int k = 0; k < NG; ++k) tot += red[k][t];
    kq[t] = tot * (1.0f / float(units));
  }
  __syncthreads();
  float a = 0.f;
  if (live) {
#pragma unroll
    for (int d = 0; d < DH; ++d) a = fmaf(wv[d], kq[DH * hf + d], a);
    if (hf == 1) half1[o] = a;
  }
  __syncthreads();
  if (hf == 1) return;
  if (live) {
    a = (bias + a) + half1[o];
    (isv ? base + z.off_vp() : base + z.off_kp())[int64_t(key) * HC + (o & (HC - 1))] = a;
  }
  uint16_t *kf = reinterpret_cast<uint16_t *>(base + z.off_kvf());
  res_kv_frag_store(kf, kf + KVF_BF16 / 2, key, o, a);
}

}  // namespace ikv
