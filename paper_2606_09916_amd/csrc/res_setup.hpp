// Per-session set-up of the residual head (Eqs. 4-6): mbar from its partial sums and the
// list of live query positions. Shared by the stand-alone set-up kernel and by the
// workgroup that the row-statistics launch adds for it.
#pragma once
#include "ikv_internal.hpp"

namespace ikv {

// Session b: mbar (from the partial sums: MBAR_PARTS row ranges, or with `pairs` one
// per head pair) and the live query positions in order. Needs at least 256 threads;
// threads past 256 only meet the barriers. Every thread of the workgroup must call it.
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
  float *misc = base + z.off_misc();
  float *mbar = misc + int64_t(MBAR_PARTS) * D;
  int *qlist = reinterpret_cast<int *>(base + z.off_qlist());
  const int t = threadIdx.x;
  {
    // 256 / D threads per channel, eight partials in flight each, merged in a fixed order
    constexpr int TPC = 256 / D;
    __shared__ float red[TPC][D];
    const float *parts = pairs ? base + z.off_mbp() : misc;
    const int np = pairs ? units / 2 : MBAR_PARTS;
    const int c = t % D, grp = t / D;
    if (t < 256) {
      float a = 0.f;
      for (int p0 = grp; p0 < np; p0 += 8 * TPC) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = parts[int64_t(min(p0 + q * TPC, np - 1)) * D + c];
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (p0 + q * TPC < np) a += v[q];
      }
      red[grp][c] = a;
    }
    __syncthreads();
    if (t < D) {
      float tot = 0.f;
#pragma unroll
      for (int k = 0; k < TPC; ++k) tot += red[k][t];
      mbar[t] = tot / float(int64_t(units) * s.R);
    }
  }
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

}  // namespace ikv
