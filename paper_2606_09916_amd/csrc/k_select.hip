// Budgeted selection of Eq. 1 (Appendix H: K = F u topk(A, max(0, C - |F|))) and
// the slot-map redirect of Eq. 7 with the alias-aware free of Sec. 3.4.
//
// Both run one 1024-thread workgroup per session: a session's positions are a
// few hundred KB at most, and every step here is integer work or a comparison.
// Order-dependent steps (the tie fill of the selection, the live and freed lists)
// give each wave one contiguous range of positions (or slot words): inside a wave
// a ballot ranks the lanes, so the workgroup needs one cross-wave scan per sweep.
#include <math.h>

#include <stdlib.h>

#include <unistd.h>

#include <atomic>
#include <mutex>
#include <chrono>
#include <random>

#include "ikv_internal.hpp"

namespace ikv {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / WAVE;
constexpr int SEL_BINS = 2048;             // radix passes of 11, 11 and 10 bits
constexpr int SEL_U = 8;                   // loads in flight per thread: every sweep is latency-bound
constexpr int SEL_CHUNK = 4096;            // positions per workgroup of k_select_keys / k_select_mark
constexpr int SEL_PART = SEL_BINS + 64;    // workspace words per chunk: histogram, counts, padding
constexpr int SEL_LIST = 16384;            // keys (with positions) of the threshold bin held in LDS
constexpr int SEL_TIES = 1024;             // ties at the threshold ranked directly (else by radix passes)

__device__ __forceinline__ uint64_t lanes_below() { return (uint64_t(1) << (threadIdx.x & 63)) - 1; }

// Loads of a batch are issued unconditionally, from an index clamped into [0, n), and
// masked afterwards: a load under a branch is waited on at once, inside the branch.
template <typename T>
__device__ __forceinline__ T ld_clamped(const T *p, int64_t i, int64_t n) {
  return p[i < n ? i : n - 1];
}

// Sum over the workgroup; `red` holds SEL_WAVES ints. Every thread must call it.
__device__ __forceinline__ int block_sum(int v, int *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int tot = 0;
#pragma unroll
  for (int w = 0; w < SEL_WAVES; ++w) tot += red[w];
  __syncthreads();
  return tot;
}

// Exclusive prefix of per-wave totals (lane 0 of each wave passes its wave's total);
// every thread gets its wave's base and the workgroup total. Every thread must call it.
__device__ __forceinline__ int wave_base(int wave_total, int &total, int *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = wave_total;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SEL_WAVES; ++w) {
    const int c = red[w];
    base += w < wave ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return base;
}

// Contiguous position range of a wave: a multiple of 64 positions per wave.
__device__ __forceinline__ void wave_range(int64_t n, int64_t &lo, int64_t &hi) {
  const int64_t seg = cdiv(cdiv(n, SEL_WAVES), WAVE) * WAVE;
  lo = min(n, int64_t(threadIdx.x >> 6) * seg);
  hi = min(n, lo + seg);
}

// Order-preserving map of a score to an unsigned key: larger score, larger key.
// NaN is ranked as -inf and -0.0 as +0.0. No score maps to 0, which marks
// "not a candidate" below.
__device__ __forceinline__ uint32_t score_key(float f) {
  if (f != f) f = -INFINITY;
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_score(uint32_t k) {
  const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

// hist[bin] += 1 for every lane with `on`. Lanes that share a bin are counted by
// their leader with one atomic (scores cluster in a few bins); after four rounds,
// or once a round finds at most two lanes on its bin, the rest add individually.
__device__ __forceinline__ void hist_add(uint32_t *hist, uint32_t bin, bool on) {
  const int lane = threadIdx.x & 63;
  uint64_t act = __ballot(on);
#pragma unroll
  for (int r = 0; r < 4 && act; ++r) {
    const int leader = __ffsll((unsigned long long)act) - 1;
    const uint32_t lb = uint32_t(__builtin_amdgcn_readlane(int(bin), leader));
    const uint64_t same = __ballot(on && bin == lb) & act;
    if (lane == leader) atomicAdd(&hist[lb], uint32_t(__popcll(same)));
    act &= ~same;
    if (__popcll(same) <= 2) break;                   // the bins are spread: no more rounds
  }
  if ((act >> lane) & 1u) atomicAdd(&hist[bin], 1u);
}

// ---- selection in three launches. Workspace, per call:
//   parts: per session and chunk of SEL_CHUNK positions, the chunk's 2048-bin
//          histogram of the top 11 key bits, its live count and live forced count;
//   keys:  the key of every position of every session at slot_off (0: not a candidate);
//   res:   per session the threshold key and the last tied position that is kept.
//   k_select_keys:   one workgroup per chunk: keys, initial keep (live forced positions,
//                    or every live position when the step is skipped), chunk histogram;
//   k_select_finish: one workgroup per session: the histograms summed, the keys of the
//                    bin that holds the take-th largest gathered with their positions,
//                    the exact threshold by radix passes over them, and among the keys
//                    equal to it the position of the last one taken (radix select on
//                    positions, smallest first);
//   k_select_mark:   one workgroup per chunk: keep every candidate above the threshold
//                    and every tie at or before that position.
__host__ __device__ inline int64_t sel_chunks_before(const ikv_session *sess, int b) {
  int64_t c = 0;
  for (int i = 0; i < b; ++i) c += cdiv(sess[i].N, SEL_CHUNK);
  return c;
}

__global__ void __launch_bounds__(256) k_select_keys(const ikv_session *__restrict__ sess,
                                                     const int32_t *__restrict__ slot_maps, int dead,
                                                     const float *__restrict__ scores, uint8_t *__restrict__ keep,
                                                     uint32_t *__restrict__ ws, int64_t keys_off) {
  __shared__ uint32_t hist[SEL_BINS];
  __shared__ int cnt[2];
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  const int64_t j0 = int64_t(blockIdx.x) * SEL_CHUNK;
  if (j0 >= s.N) return;
  const int t = threadIdx.x;
  const bool skip = s.N <= s.C;
  uint32_t *part = ws + (sel_chunks_before(sess, b) + blockIdx.x) * SEL_PART;
  uint32_t *keys = ws + keys_off + s.slot_off;
  const int32_t *S = slot_maps + s.slot_off;
  const float *sc = scores + s.slot_off;
  uint8_t *kp = keep + s.slot_off;
  for (int i = t; i < SEL_BINS; i += 256) hist[i] = 0u;
  if (t < 2) cnt[t] = 0;
  __syncthreads();
  constexpr int PER = SEL_CHUNK / 256;
  int sv[PER];
  float fv[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int64_t j = j0 + q * 256 + t;
    sv[q] = ld_clamped(S, j, s.N);
    fv[q] = ld_clamped(sc, j, s.N);
  }
  int nl = 0, nf = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int64_t j = j0 + q * 256 + t;
    const bool in = j < s.N;
    const bool live = in && sv[q] != dead;
    const bool forced = j < s.pi || (j >= s.qs && j < s.qe);
    nl += live;
    nf += live && forced;
    const bool cand = live && !forced && !skip;
    const uint32_t key = cand ? score_key(fv[q]) : 0u;
    if (in) {
      kp[j] = (live && (forced || skip)) ? 1 : 0;
      keys[j] = key;
    }
    hist_add(hist, key >> 21, cand);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    nl += __shfl_xor(nl, o, WAVE);
    nf += __shfl_xor(nf, o, WAVE);
  }
  if ((t & 63) == 0) {
    atomicAdd(&cnt[0], nl);
    atomicAdd(&cnt[1], nf);
  }
  __syncthreads();
  for (int i = t; i < SEL_BINS; i += 256) part[i] = hist[i];
  if (t < 2) part[SEL_BINS + t] = uint32_t(cnt[t]);
}

// The bin of `hist` (nbins bins, nbins / SEL_THREADS per thread) holding the kk-th
// largest value, scanning from the top bin down; writes the bin and the rank inside
// it to sh[0], sh[1]. Every thread of the workgroup must call it.
__device__ __forceinline__ void find_bin(const uint32_t *hist, int nbins, int kk, int *red, int *sh) {
  const int t = threadIdx.x, lane = t & 63;
  const int per = nbins / SEL_THREADS;
  const int hi_bin = nbins - 1 - t * per;
  int c = 0;
  for (int q = 0; q < per; ++q) c += int(hist[hi_bin - q]);
  int x = c;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, WAVE);
    if (lane >= o) x += y;
  }
  int tot;
  const int above = wave_base(__shfl(x, 63, WAVE), tot, red) + x - c;
  if (above < kk && kk <= above + c) {
    int cum = above;
    for (int q = 0; q < per; ++q) {
      const int h = int(hist[hi_bin - q]);
      if (cum + h >= kk) {
        sh[0] = hi_bin - q;
        sh[1] = kk - cum;
        break;
      }
      cum += h;
    }
  }
  __syncthreads();
}

// The kk-th largest of n values (1 <= kk <= n), get(i) -> (value, counted): radix
// passes of 11, 11 and 10 bits from the top, starting at pass p0 when the bits above
// it are already known to be `prefix` for every counted value. Every thread must call it.
template <class Get>
__device__ uint32_t kth_largest(Get get, int n, int kk, uint32_t *hist, int *red, int *sh, int p0 = 0,
                                uint32_t prefix = 0) {
  const int t = threadIdx.x;
  for (int pass = p0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const uint32_t nbins = pass == 2 ? 1024u : 2048u;
    const uint32_t himask = pass == 0 ? 0u : (0xffffffffu << (shift + (pass == 1 ? 11 : 10)));
    for (int i = t; i < SEL_BINS; i += SEL_THREADS) hist[i] = 0u;
    __syncthreads();
    for (int c0 = 0; c0 < n; c0 += SEL_THREADS * SEL_U) {
      uint32_t v[SEL_U];
      bool c[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) {
        const int i = c0 + u * SEL_THREADS + t;
        get(i < n ? i : n - 1, v[u], c[u]);
      }
#pragma unroll
      for (int u = 0; u < SEL_U; ++u)
        if (c0 + u * SEL_THREADS + t >= n) c[u] = false;
#pragma unroll
      for (int u = 0; u < SEL_U; ++u)
        hist_add(hist, (v[u] >> shift) & (nbins - 1u), c[u] && (v[u] & himask) == (prefix & himask));
    }
    __syncthreads();
    find_bin(hist, int(nbins), kk, red, sh);
    prefix |= uint32_t(sh[0]) << shift;
    kk = sh[1];
    __syncthreads();
  }
  return prefix;
}

__global__ void __launch_bounds__(SEL_THREADS) k_select_finish(const ikv_session *__restrict__ sess,
                                                               int32_t *__restrict__ n_keep, float *__restrict__ tau,
                                                               uint32_t *__restrict__ ws, int64_t keys_off,
                                                               int64_t res_off) {
  __shared__ uint32_t lkey[SEL_LIST];                 // keys of the threshold's top bin
  __shared__ uint32_t lpos[SEL_LIST];                 // their positions
  __shared__ uint32_t hist[SEL_BINS];
  __shared__ int red[SEL_WAVES];
  __shared__ int sh[2];
  __shared__ int sh_n, sh_cnt[2];
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x, lane = t & 63;
  const int64_t nch = cdiv(s.N, SEL_CHUNK);
  const uint32_t *parts = ws + sel_chunks_before(sess, b) * SEL_PART;
  const uint32_t *keys = ws + keys_off + s.slot_off;
  uint32_t *res = ws + res_off + int64_t(b) * 4;
  // chunk histograms and counts summed
  if (t < 2) sh_cnt[t] = 0;
  __syncthreads();
  for (int i = t; i < SEL_BINS + 2; i += SEL_THREADS) {
    uint32_t a = 0;
    for (int64_t c0 = 0; c0 < nch; c0 += SEL_U) {
      uint32_t v[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) v[u] = parts[(c0 + u < nch ? c0 + u : nch - 1) * SEL_PART + i];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) a += c0 + u < nch ? v[u] : 0u;
    }
    if (i < SEL_BINS) hist[i] = a;
    else sh_cnt[i - SEL_BINS] = int(a);
  }
  __syncthreads();
  const int nl = sh_cnt[0], nf = sh_cnt[1];
  const int take = s.N <= s.C ? 0 : min(max(0, s.C - nf), nl - nf);
  if (take <= 0) {                                    // nothing to rank: the keys pass left keep final
    if (t == 0) {
      n_keep[b] = s.N <= s.C ? nl : nf;
      tau[b] = s.N <= s.C ? -INFINITY : INFINITY;
      res[0] = 0xffffffffu;                           // above every key: the mark pass keeps nothing more
      res[1] = 0u;
    }
    return;
  }
  find_bin(hist, SEL_BINS, take, red, sh);
  uint32_t prefix = uint32_t(sh[0]) << 21;            // the top 11 bits of the threshold
  int kk = sh[1];                                     // its rank among the keys that share them
  int cnt = int(hist[sh[0]]);
  int level = 1;                                      // radix passes done
  __syncthreads();
  if (cnt > SEL_LIST) {
    // scores concentrate: one more pass, bits 20..10, over the keys of the bin
    for (int i = t; i < SEL_BINS; i += SEL_THREADS) hist[i] = 0u;
    __syncthreads();
    for (int c0 = 0; c0 < s.N; c0 += SEL_THREADS * SEL_U) {
      uint32_t kv[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) kv[u] = ld_clamped(keys, c0 + u * SEL_THREADS + t, s.N);
#pragma unroll
      for (int u = 0; u < SEL_U; ++u)
        hist_add(hist, (kv[u] >> 10) & 2047u,
                 c0 + u * SEL_THREADS + t < s.N && kv[u] != 0u && (kv[u] >> 21) == (prefix >> 21));
    }
    __syncthreads();
    find_bin(hist, SEL_BINS, kk, red, sh);
    prefix |= uint32_t(sh[0]) << 10;
    kk = sh[1];
    cnt = int(hist[sh[0]]);
    level = 2;
    __syncthreads();
  }
  const uint32_t known = level == 1 ? 0xffe00000u : 0xfffffc00u;   // bits fixed by the passes done
  uint32_t thr, tpos;
  if (cnt <= SEL_LIST) {
    // gather the keys that share those bits, with their positions (any order)
    if (t == 0) sh_n = 0;
    __syncthreads();
    for (int c0 = 0; c0 < s.N; c0 += SEL_THREADS * SEL_U) {
      uint32_t kv[SEL_U];
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) kv[u] = ld_clamped(keys, c0 + u * SEL_THREADS + t, s.N);
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) {
        const bool m = c0 + u * SEL_THREADS + t < s.N && kv[u] != 0u && (kv[u] & known) == prefix;
        const uint64_t bal = __ballot(m);
        int base = 0;
        if (lane == 0 && bal) base = atomicAdd(&sh_n, __popcll(bal));
        base = __shfl(base, 0, WAVE);
        if (m) {
          const int at = base + __popcll(bal & lanes_below());
          lkey[at] = kv[u];
          lpos[at] = uint32_t(c0 + u * SEL_THREADS + t);
        }
      }
    }
    __syncthreads();
    const int n = sh_n;
    thr = kth_largest([&](int i, uint32_t &v, bool &c) { v = lkey[i]; c = true; }, n, kk, hist, red, sh, level,
                      prefix);
    // keys above the threshold among them, then the ties kept: the smallest positions
    int gt = 0, eq = 0;
    for (int i = t; i < n; i += SEL_THREADS) {
      gt += lkey[i] > thr;
      eq += lkey[i] == thr;
    }
    gt = block_sum(gt, red);
    eq = block_sum(eq, red);
    const int kt = kk - gt;                           // ties taken, 1 <= kt <= eq
    if (eq <= SEL_TIES) {
      // few ties: list their positions, and the one with kt - 1 smaller ones is the last taken
      uint32_t *tie = hist;                           // the histogram is free again
      if (t == 0) sh_n = 0;
      __syncthreads();
      for (int i0 = 0; i0 < n; i0 += SEL_THREADS) {
        const int i = i0 + t;
        const bool m = i < n && lkey[i] == thr;
        const uint64_t bal = __ballot(m);
        int base = 0;
        if (lane == 0 && bal) base = atomicAdd(&sh_n, __popcll(bal));
        base = __shfl(base, 0, WAVE);
        if (m) tie[base + __popcll(bal & lanes_below())] = lpos[i];
      }
      __syncthreads();
      if (t < eq) {
        const uint32_t p = tie[t];
        int r = 0;
        for (int k = 0; k < eq; ++k) r += tie[k] < p;
        if (r == kt - 1) sh[0] = int(p);
      }
      __syncthreads();
      tpos = uint32_t(sh[0]);
    } else {
      tpos = ~kth_largest([&](int i, uint32_t &v, bool &c) { v = ~lpos[i]; c = lkey[i] == thr; }, n, kt, hist, red,
                          sh);
    }
  } else {
    // heavy ties even after 22 bits: the remaining passes and the tie order over every key
    thr = kth_largest([&](int i, uint32_t &v, bool &c) { v = keys[i]; c = v != 0u; }, s.N, kk, hist, red, sh, level,
                      prefix);
    int gt = 0;
    for (int i = t; i < s.N; i += SEL_THREADS) gt += keys[i] > thr;
    gt = block_sum(gt, red);
    tpos = ~kth_largest([&](int i, uint32_t &v, bool &c) { c = keys[i] == thr; v = ~uint32_t(i); }, s.N, take - gt,
                        hist, red, sh);
  }
  if (t == 0) {
    res[0] = thr;
    res[1] = tpos;
    n_keep[b] = nf + take;
    tau[b] = key_score(thr);
  }
}

__global__ void __launch_bounds__(256) k_select_mark(const ikv_session *__restrict__ sess, uint8_t *__restrict__ keep,
                                                     const uint32_t *__restrict__ ws, int64_t keys_off,
                                                     int64_t res_off) {
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  const int64_t j0 = int64_t(blockIdx.x) * SEL_CHUNK;
  if (j0 >= s.N) return;
  const uint32_t thr = ws[res_off + int64_t(b) * 4], tpos = ws[res_off + int64_t(b) * 4 + 1];
  if (thr == 0xffffffffu) return;
  const uint32_t *keys = ws + keys_off + s.slot_off;
  uint8_t *kp = keep + s.slot_off;
  constexpr int PER = SEL_CHUNK / 256;
  uint32_t kv[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) kv[q] = ld_clamped(keys, j0 + q * 256 + threadIdx.x, int64_t(s.N));
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int64_t j = j0 + q * 256 + threadIdx.x;
    if (j < s.N && (kv[q] > thr || (kv[q] == thr && uint32_t(j) <= tpos))) kp[j] = 1;
  }
}

// ---- selection in one launch for sessions of at most SEL_SMALL positions: one
// workgroup per session holds every key in LDS, so the radix passes and the tie
// ranking never leave the CU. Thread t takes positions t + 1024 q; wave w's 64
// consecutive positions of sweep q give one 64-bit ballot of the initial keep flags.
// Scores concentrate in a narrow range, so the passes bin the keys still in play,
// [lo, hi], by their offset from lo: 11 bits of the actual spread per pass.
constexpr int SEL_SMALL = 32768;
constexpr int SEL_SU = 32;                 // loads in flight per thread while the keys are read

__device__ __forceinline__ uint32_t block_min(uint32_t v, int *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, uint32_t(__shfl_xor(int(v), o, WAVE)));
  if (lane == 0) red[wave] = int(v);
  __syncthreads();
  uint32_t r = 0xffffffffu;
#pragma unroll
  for (int w = 0; w < SEL_WAVES; ++w) r = min(r, uint32_t(red[w]));
  __syncthreads();
  return r;
}

__global__ void __launch_bounds__(SEL_THREADS) k_select_small(const ikv_session *__restrict__ sess,
                                                              const int32_t *__restrict__ slot_maps, int dead,
                                                              const float *__restrict__ scores,
                                                              uint8_t *__restrict__ keep, int32_t *__restrict__ n_keep,
                                                              float *__restrict__ tau) {
  __shared__ uint32_t keys[SEL_SMALL];                // 0: not a candidate
  __shared__ uint64_t kbits[SEL_SMALL / 64];          // live forced positions (every live one when skipped)
  __shared__ uint32_t hist[SEL_BINS];
  __shared__ int red[SEL_WAVES];
  __shared__ int sh[2];
  constexpr int Q = SEL_SMALL / SEL_THREADS;
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x, lane = t & 63;
  const int N = s.N;
  const bool skip = N <= s.C;
  const int32_t *S = slot_maps + s.slot_off;
  const float *sc = scores + s.slot_off;
  uint8_t *kp = keep + s.slot_off;
  int nl = 0, nf = 0;
  uint32_t kmin = 0xffffffffu, kmax = 0u;             // over the candidates
  for (int q0 = 0; q0 < Q; q0 += SEL_SU) {
    if (q0 * SEL_THREADS >= N) break;
    int sv[SEL_SU];
    float fv[SEL_SU];
#pragma unroll
    for (int u = 0; u < SEL_SU; ++u) {
      const int j = (q0 + u) * SEL_THREADS + t;
      sv[u] = ld_clamped(S, j, N);
      fv[u] = ld_clamped(sc, j, N);
    }
#pragma unroll
    for (int u = 0; u < SEL_SU; ++u) {
      const int j = (q0 + u) * SEL_THREADS + t;
      const bool in = j < N;
      const bool live = in && sv[u] != dead;
      const bool forced = j < s.pi || (j >= s.qs && j < s.qe);
      nl += live;
      nf += live && forced;
      const bool cand = live && !forced && !skip;
      const uint32_t key = cand ? score_key(fv[u]) : 0u;
      keys[j] = key;
      if (cand) {
        kmin = min(kmin, key);
        kmax = max(kmax, key);
      }
      const uint64_t kb = __ballot(live && (forced || skip));
      if (lane == 0) kbits[j >> 6] = kb;
    }
  }
  nl = block_sum(nl, red);
  nf = block_sum(nf, red);
  const int take = skip ? 0 : min(max(0, s.C - nf), nl - nf);
  uint32_t thr = 0xffffffffu, tpos = 0u;              // above every key: nothing beyond the initial keep
  if (take > 0) {
    // the take-th largest key: shrink [lo, hi] until it holds one value
    uint32_t lo = block_min(kmin, red), hi = ~block_min(~kmax, red);
    int kk = take;                                    // its rank from the top among keys in [lo, hi]
    const int n = min(N, SEL_SMALL);
    while (hi > lo) {
      const int span = 32 - __clz(int(hi - lo));      // bits of hi - lo
      const int shift = max(0, span - 11);
      for (int i = t; i < SEL_BINS; i += SEL_THREADS) hist[i] = 0u;
      __syncthreads();
      for (int i0 = 0; i0 < n; i0 += SEL_THREADS * SEL_U) {
        uint32_t kv[SEL_U];
#pragma unroll
        for (int u = 0; u < SEL_U; ++u) kv[u] = keys[min(i0 + u * SEL_THREADS + t, n - 1)];
#pragma unroll
        for (int u = 0; u < SEL_U; ++u) {
          const bool on = i0 + u * SEL_THREADS + t < n && kv[u] >= lo && kv[u] <= hi;
          hist_add(hist, on ? (kv[u] - lo) >> shift : 0u, on);
        }
      }
      __syncthreads();
      find_bin(hist, SEL_BINS, kk, red, sh);
      const uint32_t nlo = lo + (uint32_t(sh[0]) << shift);
      hi = shift == 0 ? nlo : min(hi, nlo + ((1u << shift) - 1u));
      lo = nlo;
      kk = sh[1];
      __syncthreads();
    }
    thr = lo;
    int gt = 0, eq = 0;
    for (int i = t; i < n; i += SEL_THREADS) {
      gt += keys[i] > thr;
      eq += keys[i] == thr;
    }
    gt = block_sum(gt, red);
    eq = block_sum(eq, red);
    const int kt = take - gt;                         // ties taken, 1 <= kt <= eq
    // all ties taken: any position passes; else the kt-th smallest tied position
    tpos = kt == eq ? 0xffffffffu
                    : ~kth_largest([&](int i, uint32_t &v, bool &c) { v = ~uint32_t(i); c = keys[i] == thr; }, n, kt,
                                   hist, red, sh);
  }
  for (int q = 0; q < Q; ++q) {
    const int j = q * SEL_THREADS + t;
    if (j >= N) break;
    const uint32_t k = keys[j];
    const bool sel = k != 0u && (k > thr || (k == thr && uint32_t(j) <= tpos));
    kp[j] = uint8_t(sel || ((kbits[j >> 6] >> lane) & 1u));
  }
  if (t == 0) {
    n_keep[b] = skip ? nl : nf + take;
    tau[b] = skip ? -INFINITY : (take > 0 ? key_score(thr) : INFINITY);
  }
}

// ---- selection across workgroups (a cooperative launch: every workgroup of the grid
// is resident at once). Each session's positions split into chunks of SC_CHUNK, one
// workgroup each, holding its keys in LDS; the workgroups of a session meet at
// barriers on flags in the workspace. Counts and key range go through per-workgroup
// partials, the radix histograms are summed with integer device-scope atomics
// (order-free, so the result is deterministic), and every workgroup then takes the same
// decisions from the same totals: the passes bin the keys still in play by their
// offset from the smallest candidate key, 11 bits of the actual spread per pass; ties
// at the threshold are ranked by the same passes over positions. Nothing in the
// workspace needs to be cleared beforehand: each workgroup clears its share of the
// histograms before the first barrier, and the barrier flags carry a stamp that the
// host draws afresh for every call (above every earlier call's, with a random tag per
// process in the top bits, so that no structured leftover in the workspace matches).
// The barrier polls a bounded number of times; a workgroup whose poll runs out sets a
// fault word in pinned host memory, which the library's next call turns into IKV_EHIP:
// the kept set of the call that timed out is not valid.
constexpr int SC_THREADS = 256;
constexpr int SC_WAVES = SC_THREADS / WAVE;
constexpr int SC_PER = 4;                              // positions per thread
constexpr int SC_CHUNK = SC_THREADS * SC_PER;
constexpr int SC_MAXN = 131072;                        // positions per session on this path
constexpr int SC_MAXG = SC_MAXN / SC_CHUNK;            // workgroups per session
constexpr int SC_HIST = 5;                             // histograms: 3 key passes, 2 position passes
constexpr int SC_BARS = 8;                             // stamps per call (at most 1 + 5 barriers)
// per session: a 64-bit barrier flag per workgroup, four partial words per workgroup
// (live count, live forced count, ~(min key), max key), then the histograms
constexpr int SC_PART = 2 * SC_MAXG;
constexpr int SC_HIST0 = SC_PART + 4 * SC_MAXG;
constexpr int SC_WORDS = SC_HIST0 + SC_HIST * SEL_BINS;
static_assert(SC_MAXG <= 2 * WAVE, "the barrier poll reads at most two flags per lane");

__device__ __forceinline__ uint32_t ald(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void ast(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void aadd(uint32_t *p, uint32_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Barrier of a session's G workgroups, stamped `stamp`: workgroup wg sets its flag to
// the stamp and waits until every flag of the session lies in [stamp, last], the
// stamps of this barrier and of the call's later ones (a workgroup may already have
// moved on). The host draws the call's stamps above every earlier call's, so a flag
// left by an earlier call never passes, and puts a random per-process tag in the top
// 24 bits, so that leftovers of other calls (counts, bitsets, floats) pass only by
// matching both the tag and an 8-stamp window. Everything the workgroups exchange is a
// device-scope atomic, so the barrier needs no cache write-back or invalidation: each
// thread's atomics are complete once its vector-memory count drains, then one thread
// sets the flag and one wave polls the flags with coherent loads. Every workgroup of
// the grid is resident (cooperative launch), so every flag is set; the poll is bounded
// all the same (`spins` polls), and a poll that runs out sets `timed_out` and lets the
// workgroup go on.
__device__ __forceinline__ void sc_barrier(uint64_t *flags, int G, int wg, uint64_t stamp, uint64_t last,
                                           uint32_t spins, int *sh_ok, bool &timed_out) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const int t = threadIdx.x;
  if (t < WAVE) {
    if (t == 0) __hip_atomic_store(flags + wg, stamp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bool done = false;
    for (uint32_t spin = 0; spin < spins; ++spin) {
      bool ok = true;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int j = t + k * WAVE;
        if (j < G) {
          const uint64_t f = __hip_atomic_load(flags + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ok = ok && f >= stamp && f <= last;
        }
      }
      if (__all(ok)) {
        done = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (t == 0) *sh_ok = done;
  }
  __syncthreads();
  timed_out = timed_out || !*sh_ok;
}

// Sum and maximum over the workgroup of SC_THREADS threads.
__device__ __forceinline__ uint32_t sc_umax(uint32_t v, int *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, uint32_t(__shfl_xor(int(v), o, WAVE)));
  if (lane == 0) red[wave] = int(v);
  __syncthreads();
  uint32_t r = 0u;
#pragma unroll
  for (int w = 0; w < SC_WAVES; ++w) r = max(r, uint32_t(red[w]));
  __syncthreads();
  return r;
}

__device__ __forceinline__ int sc_sum(int v, int *red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int tot = 0;
#pragma unroll
  for (int w = 0; w < SC_WAVES; ++w) tot += red[w];
  __syncthreads();
  return tot;
}

// The bin of the session histogram `gh` holding the kk-th largest (scanning from the
// top bin); copies the histogram into `lh` and writes the bin and the rank inside it
// to sh[0], sh[1]. Every thread must call it.
__device__ __forceinline__ void sc_find_bin(const uint32_t *gh, uint32_t *lh, int kk, int *red, int *sh) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  if (t == 0) {          // no bin holds rank kk only if the histograms are not whole (a timed-out barrier)
    sh[0] = 0;
    sh[1] = 1;
  }
  constexpr int per = SEL_BINS / SC_THREADS;
  const int hi_bin = SEL_BINS - 1 - t * per;
  uint32_t v[per];
#pragma unroll
  for (int q = 0; q < per; ++q) v[q] = ald(gh + hi_bin - q);
  int c = 0;
#pragma unroll
  for (int q = 0; q < per; ++q) {
    lh[hi_bin - q] = v[q];
    c += int(v[q]);
  }
  int x = c;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, WAVE);
    if (lane >= o) x += y;
  }
  if (lane == 63) red[wave] = x;
  __syncthreads();
  int base = 0;
#pragma unroll
  for (int w = 0; w < SC_WAVES; ++w) base += w < wave ? red[w] : 0;
  const int above = base + x - c;
  if (above < kk && kk <= above + c) {
    int cum = above;
#pragma unroll
    for (int q = 0; q < per; ++q) {
      const int h = int(v[q]);
      if (cum < kk && cum + h >= kk) {
        sh[0] = hi_bin - q;
        sh[1] = kk - cum;
      }
      cum += h;
    }
  }
  __syncthreads();
}

// The kk-th largest of this chunk's values get(i) among those counted, merged with
// the session's other chunks: [lo, hi] holds it and kk is its rank from the top among
// the values in [lo, hi]; pass p uses histogram hist0 + p. Every workgroup of the
// session calls it with the same arguments and takes the same passes. Returns the
// value; *cnt is the number of counted values equal to it.
template <class Get>
__device__ uint32_t sc_kth(Get get, uint32_t lo, uint32_t hi, int kk, uint32_t *cw, int hist0, uint32_t *lh,
                           int *red, int *sh, uint64_t &stamp, uint64_t last, int G, int wg, int &cnt,
                           uint32_t spins, bool &timed_out) {
  const int t = threadIdx.x;
  int pass = 0;
  cnt = -1;
  while (hi > lo) {
    const int span = 32 - __clz(int(hi - lo));
    const int shift = max(0, span - 11);
    for (int i = t; i < SEL_BINS; i += SC_THREADS) lh[i] = 0u;
    __syncthreads();
#pragma unroll
    for (int q = 0; q < SC_PER; ++q) {
      uint32_t v;
      bool c;
      get(q * SC_THREADS + t, v, c);
      const bool on = c && v >= lo && v <= hi;
      hist_add(lh, on ? (v - lo) >> shift : 0u, on);
    }
    __syncthreads();
    uint32_t *gh = cw + SC_HIST0 + (hist0 + pass) * SEL_BINS;
    for (int i = t; i < SEL_BINS; i += SC_THREADS)
      if (lh[i]) aadd(gh + i, lh[i]);
    sc_barrier(reinterpret_cast<uint64_t *>(cw), G, wg, ++stamp, last, spins, sh + 2, timed_out);
    sc_find_bin(gh, lh, kk, red, sh);
    const uint32_t nlo = lo + (uint32_t(sh[0]) << shift);
    hi = shift == 0 ? nlo : min(hi, nlo + ((1u << shift) - 1u));
    lo = nlo;
    kk = sh[1];
    cnt = int(lh[min(sh[0], SEL_BINS - 1)]);
    ++pass;
    __syncthreads();
  }
  return lo;
}

__global__ void __launch_bounds__(SC_THREADS) k_select_coop(const ikv_session *__restrict__ sess,
                                                            const int32_t *__restrict__ slot_maps, int dead,
                                                            const float *__restrict__ scores,
                                                            uint8_t *__restrict__ keep, int32_t *__restrict__ n_keep,
                                                            float *__restrict__ tau, uint32_t *__restrict__ coop,
                                                            uint64_t stamp0, uint32_t spins,
                                                            uint32_t *__restrict__ host_fault) {
  __shared__ uint32_t ck[SC_CHUNK];                  // keys of this chunk (0: not a candidate)
  __shared__ uint32_t lh[SEL_BINS];
  __shared__ int red[SC_WAVES];
  __shared__ int sh[3];                              // bin, rank within it; barrier outcome
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  const int N = s.N;
  const int G = max(1, int(cdiv(N, SC_CHUNK)));     // an empty session still writes its counts
  const int wg = blockIdx.x;
  if (wg >= G) return;                               // not one of this session's workgroups
  const int t = threadIdx.x;
  uint32_t *cw = coop + int64_t(b) * SC_WORDS;
  const bool skip = N <= s.C;
  const int j0 = wg * SC_CHUNK;
  const int32_t *S = slot_maps + s.slot_off;
  const float *sc = scores + s.slot_off;
  uint8_t *kp = keep + s.slot_off;

  // keys, initial keep flags (live forced, or every live position when skipped), counts, key range
  int sv[SC_PER];
  float fv[SC_PER];
#pragma unroll
  for (int q = 0; q < SC_PER; ++q) {
    const int j = j0 + q * SC_THREADS + t;
    sv[q] = ld_clamped(S, j, N);
    fv[q] = ld_clamped(sc, j, N);
  }
  int nl = 0, nf = 0;
  uint32_t nmin = 0u, kmax = 0u, kflag = 0u;         // nmin: complement of the smallest key
#pragma unroll
  for (int q = 0; q < SC_PER; ++q) {
    const int j = j0 + q * SC_THREADS + t;
    const bool live = j < N && sv[q] != dead;
    const bool forced = j < s.pi || (j >= s.qs && j < s.qe);
    nl += live;
    nf += live && forced;
    const bool cand = live && !forced && !skip;
    const uint32_t key = cand ? score_key(fv[q]) : 0u;
    ck[q * SC_THREADS + t] = key;
    kflag |= uint32_t(live && (forced || skip)) << q;
    if (cand) {
      nmin = max(nmin, ~key);
      kmax = max(kmax, key);
    }
  }
  nl = sc_sum(nl, red);
  nf = sc_sum(nf, red);
  nmin = sc_umax(nmin, red);
  kmax = sc_umax(kmax, red);
  uint32_t *part = cw + SC_PART;
  if (t < 4) ast(part + 4 * wg + t, t == 0 ? uint32_t(nl) : t == 1 ? uint32_t(nf) : t == 2 ? nmin : kmax);
  // this workgroup's share of the session's histograms starts at zero
  for (int i = wg * SC_THREADS + t; i < SC_HIST * SEL_BINS; i += G * SC_THREADS) ast(cw + SC_HIST0 + i, 0u);
  uint64_t stamp = stamp0;
  const uint64_t last = stamp + SC_BARS - 1;
  bool timed_out = false;
  sc_barrier(reinterpret_cast<uint64_t *>(cw), G, wg, ++stamp, last, spins, sh + 2, timed_out);
  // the session's totals from every workgroup's partials (the same in every workgroup)
  uint32_t p0 = 0u, p1 = 0u, p2 = 0u, p3 = 0u;
  if (t < G) {
    p0 = ald(part + 4 * t);
    p1 = ald(part + 4 * t + 1);
    p2 = ald(part + 4 * t + 2);
    p3 = ald(part + 4 * t + 3);
  }
  const int tl = sc_sum(int(p0), red), tf = sc_sum(int(p1), red);
  const uint32_t lo_key = ~sc_umax(p2, red), hi_key = sc_umax(p3, red);
  const int take = skip ? 0 : min(max(0, s.C - tf), tl - tf);
  uint32_t thr = 0xffffffffu, tpos = 0u;             // above every key: nothing beyond the initial keep
  if (take > 0) {
    int cnt;
    thr = sc_kth([&](int i, uint32_t &v, bool &c) { v = ck[i]; c = v != 0u; }, lo_key, hi_key,
                 take, cw, 0, lh, red, sh, stamp, last, G, wg, cnt, spins, timed_out);
    // rank of the threshold among the keys equal to it, and how many there are
    const int eq = cnt < 0 ? tl - tf : cnt;           // no pass: every candidate has the same key
    const int kt = cnt < 0 ? take : sh[1];
    // all ties taken: any position passes; else the kt-th smallest tied position
    if (kt == eq) {
      tpos = 0xffffffffu;
    } else {
      int c2;
      tpos = ~sc_kth([&](int i, uint32_t &v, bool &c) { v = ~uint32_t(j0 + i); c = ck[i] == thr; },
                     ~uint32_t(N - 1), 0xffffffffu, kt, cw, 3, lh, red, sh, stamp, last, G, wg, c2, spins,
                     timed_out);
    }
  }
#pragma unroll
  for (int q = 0; q < SC_PER; ++q) {
    const int j = j0 + q * SC_THREADS + t;
    if (j < N) {
      const uint32_t k = ck[q * SC_THREADS + t];
      const bool sel = k != 0u && (k > thr || (k == thr && uint32_t(j) <= tpos));
      kp[j] = uint8_t(sel || ((kflag >> q) & 1u));
    }
  }
  if (wg == 0 && t == 0) {
    n_keep[b] = skip ? tl : tf + take;
    tau[b] = skip ? -INFINITY : (take > 0 ? key_score(thr) : INFINITY);
  }
  // a timed-out barrier: the host's fault word, which the library's next call reports
  if (t == 0 && timed_out && host_fault)
    __hip_atomic_store(host_fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Words before the cooperative path's block (which starts 256-byte aligned).
static int64_t select_coop_off(const ikv_session *sess, int B, int64_t total_positions) {
  return align64f(sel_chunks_before(sess, B) * SEL_PART + total_positions + int64_t(B) * 4);
}

size_t select_workspace_bytes(const ikv_session *sess, int B, int64_t total_positions) {
  return size_t(select_coop_off(sess, B, total_positions) + int64_t(B) * SC_WORDS) * sizeof(uint32_t);
}

// Polls of a grid barrier before it gives up: IKV_SELECT_SPINS in the environment
// (read on every call; a host-side way to force the give-up path in tests), else 2^24.
static uint32_t select_spin_limit() {
  const char *e = getenv("IKV_SELECT_SPINS");
  if (e == nullptr || e[0] == '\0') return 1u << 24;
  return uint32_t(strtoul(e, nullptr, 10));
}

// Workgroups a cooperative launch of k_select_coop may have on the current device
// (0: not available). IKV_NO_COOP=1 in the environment turns the cooperative path off,
// for tools that cannot follow a cooperative launch; the selection is the same.
static int coop_capacity() {
  static int cap[64];
  static bool known[64];
  const char *e = getenv("IKV_NO_COOP");           // read on every call
  if (e != nullptr && e[0] != '\0' && e[0] != '0') return 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (!known[dev]) {
    int per_cu = 0, cus = 0, coop = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_select_coop, SC_THREADS, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess)
      per_cu = cus = coop = 0;
    cap[dev] = coop ? per_cu * cus : 0;
    known[dev] = true;
  }
  return cap[dev];
}

// ---- scratch of the allocation-free selection (ikv_select_budget_static): one array
// per device, held until the process ends, shared by every call on that device. Host
// code reaches it only through the address hipGetSymbolAddress returns.
static __device__ __align__(256) uint32_t scratch[IKV_SELECT_STATIC_MAX_BYTES / 4];

namespace {
std::mutex g_scratch_mu;
uint32_t *g_scratch[64];                           // per device, resolved once with that device current
}  // namespace

hipError_t select_static_scratch(uint32_t **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<uint32_t *>(p);
  }
  *ptr = g_scratch[dev];
  return hipSuccess;
}

hipError_t launch_select(const ikv_session *sess_host, const ikv_session *sess_dev, int B, int maxN,
                         const int32_t *slot_maps, int32_t dead, const float *scores, uint8_t *keep,
                         int32_t *n_keep, float *tau, uint32_t *ws, int64_t total_positions, hipStream_t st,
                         bool may_alloc) {
  const int64_t keys_off = sel_chunks_before(sess_host, B) * SEL_PART;
  const int64_t res_off = keys_off + total_positions;
  const int64_t gmax = cdiv(maxN, SC_CHUNK);
  if (maxN > 0 && maxN <= SC_MAXN && gmax * B <= coop_capacity()) {
    uint32_t *coop = ws + select_coop_off(sess_host, B, total_positions);
    // the barrier stamps of this call: a random per-process tag in bits 40-63, above it
    // a counter of calls (2^37 calls before it wraps), SC_BARS stamps per call
    static const uint64_t tag = [] {
      std::random_device rd;
      uint64_t x = (uint64_t(rd()) << 32) ^ rd() ^ uint64_t(getpid()) ^
                   uint64_t(std::chrono::steady_clock::now().time_since_epoch().count());
      x &= 0xffffffull;
      return (x == 0 || x == 0xffffffull ? 0x5a5a5aull : x) << 40;
    }();
    static std::atomic<uint64_t> calls{1};
    uint64_t stamp0 = tag | ((calls.fetch_add(1) * SC_BARS) & ((1ull << 40) - 1));
    uint32_t spins = select_spin_limit();
    uint32_t *fault = may_alloc ? host_fault_word() : host_fault_word_if_any();
    KTimer kt_("k_select_coop", st);
    void *args[] = {(void *)&sess_dev, (void *)&slot_maps, (void *)&dead, (void *)&scores, (void *)&keep,
                    (void *)&n_keep, (void *)&tau, (void *)&coop, (void *)&stamp0, (void *)&spins, (void *)&fault};
    hipError_t e = hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k_select_coop), dim3(unsigned(gmax), B),
                                              dim3(SC_THREADS), args, 0, st);
    if (e != hipSuccess) return e;
    return hipGetLastError();
  }
  if (maxN <= SEL_SMALL) {
    KTimer kt_("k_select_small", st);
    k_select_small<<<B, SEL_THREADS, 0, st>>>(sess_dev, slot_maps, dead, scores, keep, n_keep, tau);
    return hipGetLastError();
  }
  const dim3 grid(unsigned(cdiv(maxN, SEL_CHUNK)), B);
  if (maxN > 0) {
    KTimer kt_("k_select_keys", st);
    k_select_keys<<<grid, 256, 0, st>>>(sess_dev, slot_maps, dead, scores, keep, ws, keys_off);
  }
  {
    KTimer kt_("k_select_finish", st);
    k_select_finish<<<B, SEL_THREADS, 0, st>>>(sess_dev, n_keep, tau, ws, keys_off, res_off);
  }
  if (maxN > 0) {
    KTimer kt_("k_select_mark", st);
    k_select_mark<<<grid, 256, 0, st>>>(sess_dev, keep, ws, keys_off, res_off);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ redirect
// Two slot sets: slots of kept positions, freed slots. Where they live (RED_MODE):
//   RED_BYTES (pools up to 65,536 slots): one LDS byte per slot, set by plain byte
//     stores. Every writer stores the same 1, so no atomics are needed; an LDS atomic
//     OR serialises the lanes that hit one word, and the 16 positions of a page do.
//   RED_LDS_BITS (up to RED_LDS_WORDS * 32 slots): LDS bitsets, set by atomic OR.
//   RED_GLOBAL_BITS: bitsets in the caller's workspace, where the workgroup's waves
//     reach each other through device-scope atomics and fences.
constexpr int RED_LDS_WORDS = 16384;        // two bitsets of 64 KB: pools up to 524288 slots
constexpr int RED_BYTE_SLOTS = 65536;       // two byte maps of 64 KB
constexpr int RED_U = 16;                   // positions in flight per lane in the two sweeps
enum { RED_BYTES = 0, RED_LDS_BITS = 1, RED_GLOBAL_BITS = 2 };

template <int MODE>
struct SlotSets {
  uint32_t *kept, *freed;
  __device__ __forceinline__ void set(uint32_t *w, int u) const {
    if (MODE == RED_BYTES) *reinterpret_cast<volatile uint8_t *>(reinterpret_cast<uint8_t *>(w) + u) = 1;
    else if (MODE == RED_LDS_BITS) atomicOr(w + (u >> 5), 1u << (u & 31));
    else __hip_atomic_fetch_or(w + (u >> 5), 1u << (u & 31), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // bit k of word i <-> slot 32 i + k
  __device__ __forceinline__ uint32_t word(const uint32_t *w, int64_t i) const {
    if (MODE == RED_BYTES) {
      const uint4 *p = reinterpret_cast<const uint4 *>(w) + 2 * i;
      const uint4 a = p[0], c = p[1];
      const uint32_t x[8] = {a.x, a.y, a.z, a.w, c.x, c.y, c.z, c.w};
      uint32_t m = 0;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        m |= ((x[k] & 1u) | ((x[k] >> 7) & 2u) | ((x[k] >> 14) & 4u) | ((x[k] >> 21) & 8u)) << (4 * k);
      return m;
    }
    if (MODE == RED_LDS_BITS) return w[i];
    return __hip_atomic_load(w + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __device__ __forceinline__ bool test(const uint32_t *w, int u) const {
    if (MODE == RED_BYTES) return reinterpret_cast<const uint8_t *>(w)[u] != 0;
    return (word(w, u >> 5) >> (u & 31)) & 1u;
  }
  // every word of both sets (words = 32-slot groups), cleared by the workgroup
  __device__ __forceinline__ void clear_all(int64_t words, int t) const {
    const int64_t n = MODE == RED_BYTES ? words * 8 : words;   // 32-bit stores per set
    for (int64_t i = t; i < n; i += SEL_THREADS) {
      if (MODE == RED_GLOBAL_BITS) {
        __hip_atomic_store(kept + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(freed + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {
        kept[i] = 0u;
        freed[i] = 0u;
      }
    }
  }
  __device__ __forceinline__ void sync() const {
    if (MODE == RED_GLOBAL_BITS) __threadfence();
    __syncthreads();
  }
};

template <int MODE>
__global__ void __launch_bounds__(SEL_THREADS) k_redirect(const ikv_session *__restrict__ sess, int64_t num_slots,
                                                          int32_t *__restrict__ slot_maps, int dead,
                                                          const uint8_t *__restrict__ keep, int32_t *__restrict__ freed,
                                                          int32_t *__restrict__ n_freed, int32_t *__restrict__ live,
                                                          int32_t *__restrict__ n_live, uint32_t *__restrict__ ws) {
  __shared__ __align__(16) uint32_t lds_sets[MODE != RED_GLOBAL_BITS ? 2 * RED_LDS_WORDS : 1];
  __shared__ int red[SEL_WAVES];
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x, lane = t & 63;
  int32_t *S = slot_maps + s.slot_off;
  const uint8_t *kp = keep + s.slot_off;
  const int64_t words = bitset_words(num_slots);
  SlotSets<MODE> sets;
  sets.kept = MODE != RED_GLOBAL_BITS ? lds_sets : ws + int64_t(b) * 2 * words;
  sets.freed = sets.kept + (MODE == RED_BYTES ? words * 8 : words);
  sets.clear_all(words, t);
  sets.sync();
  // slots of the kept positions, and the survivors of each wave's range
  int64_t lo, hi;
  wave_range(s.N, lo, hi);
  int surv = 0;
  for (int64_t c0 = lo; c0 < hi; c0 += WAVE * RED_U) {
    int sv[RED_U];
    uint8_t kv[RED_U];
#pragma unroll
    for (int u = 0; u < RED_U; ++u) {
      const int64_t j = c0 + u * WAVE + lane;
      sv[u] = ld_clamped(S, j, hi);
      kv[u] = ld_clamped(kp, j, hi);
    }
#pragma unroll
    for (int u = 0; u < RED_U; ++u) {
      const bool k = c0 + u * WAVE + lane < hi && sv[u] != dead && kv[u] != 0;
      if (k) sets.set(sets.kept, sv[u]);
      surv += __popcll(__ballot(k));
    }
  }
  int total_live;
  int pos = wave_base(surv, total_live, red);
  sets.sync();
  // reroute dropped positions, mark freeable slots, list the survivors in position order
  for (int64_t c0 = lo; c0 < hi; c0 += WAVE * RED_U) {
    int sv[RED_U];
    uint8_t kv[RED_U];
#pragma unroll
    for (int q = 0; q < RED_U; ++q) {
      const int64_t j = c0 + q * WAVE + lane;
      sv[q] = ld_clamped(S, j, hi);
      kv[q] = ld_clamped(kp, j, hi);
    }
#pragma unroll
    for (int q = 0; q < RED_U; ++q) {
      const int j = int(c0) + q * WAVE + lane;
      const int u = j < hi ? sv[q] : dead;
      const bool alive = u != dead;
      const bool k = alive && kv[q] != 0;
      if (alive && !k) {
        S[j] = dead;
        if (j >= s.radix_prefix && !sets.test(sets.kept, u)) sets.set(sets.freed, u);
      }
      const uint64_t bal = __ballot(k);
      if (k) live[s.slot_off + pos + __popcll(bal & lanes_below())] = u;
      pos += __popcll(bal);
    }
  }
  if (t == 0) n_live[b] = total_live;
  sets.sync();
  // freed slots in ascending slot order: wave w lists the slots of its range of words
  int64_t wlo, whi;
  wave_range(words, wlo, whi);
  int nbits = 0;
  for (int64_t i = wlo + lane; i < whi; i += WAVE) nbits += __popc(sets.word(sets.freed, i));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) nbits += __shfl_xor(nbits, o, WAVE);
  int total_freed;
  int fpos = wave_base(nbits, total_freed, red);
  // The freed slots of a step go out as one run, in slot order: lane = slot (64 per
  // step) on bitsets; with byte maps lane l takes slots 4l .. 4l+3 of the step (256
  // per step, one 32-bit LDS read), each slot's place from four ballots.
  if (MODE == RED_BYTES) {
    const uint8_t *fb = reinterpret_cast<const uint8_t *>(sets.freed);
    const uint64_t below = lanes_below();
    for (int64_t base = wlo * 32; base < whi * 32; base += 4 * WAVE) {
      const int64_t u0 = base + 4 * lane;
      const uint32_t x = u0 < whi * 32 ? *reinterpret_cast<const uint32_t *>(fb + u0) : 0u;
      const uint64_t b0 = __ballot(x & 0xffu), b1 = __ballot(x & 0xff00u), b2 = __ballot(x & 0xff0000u),
                     b3 = __ballot(x & 0xff000000u);
      int r = fpos + __popcll(b0 & below) + __popcll(b1 & below) + __popcll(b2 & below) + __popcll(b3 & below);
      int32_t *out = freed + s.slot_off;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if ((x >> (8 * k)) & 0xffu) out[r++] = int32_t(u0 + k);
      fpos += __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
    }
  } else {
    for (int64_t base = wlo * 32; base < whi * 32; base += WAVE) {
      const int64_t u = base + lane;
      const bool f = u < whi * 32 && sets.test(sets.freed, int(u));
      const uint64_t bal = __ballot(f);
      if (f) freed[s.slot_off + fpos + __popcll(bal & lanes_below())] = int32_t(u);
      fpos += __popcll(bal);
    }
  }
  if (t == 0) n_freed[b] = total_freed;
}

hipError_t launch_redirect(const ikv_session *sess_dev, int B, int64_t num_slots, int32_t *slot_maps, int32_t dead,
                           const uint8_t *keep, int32_t *freed, int32_t *n_freed, int32_t *live, int32_t *n_live,
                           uint32_t *ws, hipStream_t st) {
  if (num_slots <= RED_BYTE_SLOTS)
    {
      KTimer kt_("k_redirect<bytes>", st);
      k_redirect<RED_BYTES><<<B, SEL_THREADS, 0, st>>>(sess_dev, num_slots, slot_maps, dead, keep, freed, n_freed,
                                                       live, n_live, ws);
    }
  else if (bitset_words(num_slots) <= RED_LDS_WORDS)
    {
      KTimer kt_("k_redirect<lds>", st);
      k_redirect<RED_LDS_BITS><<<B, SEL_THREADS, 0, st>>>(sess_dev, num_slots, slot_maps, dead, keep, freed, n_freed,
                                                          live, n_live, ws);
    }
  else
    {
      KTimer kt_("k_redirect<global>", st);
      k_redirect<RED_GLOBAL_BITS><<<B, SEL_THREADS, 0, st>>>(sess_dev, num_slots, slot_maps, dead, keep, freed,
                                                             n_freed, live, n_live, ws);
    }
  return hipGetLastError();
}

}  // namespace ikv
