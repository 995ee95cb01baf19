// Budgeted selection of Eq. 1 (Appendix H: K = F u topk(A, max(0, C - |F|))) and
// the slot-map redirect of Eq. 7 with the alias-aware free of Sec. 3.4.
//
// Both run one 1024-thread workgroup per session: a session's positions are a
// few hundred KB at most, and every step here is integer work or a comparison.
// Order-dependent steps (the tie fill of the selection, the live and freed lists)
// give each wave one contiguous range of positions (or slot words): inside a wave
// a ballot ranks the lanes, so the workgroup needs one cross-wave scan per sweep.
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / WAVE;
constexpr int SEL_LDS_KEYS = 32768;        // sessions up to this N keep their keys in LDS
constexpr int SEL_BINS = 2048;             // radix passes of 11, 11 and 10 bits
constexpr int SEL_U = 8;                   // loads in flight per thread: every sweep is latency-bound

__device__ __forceinline__ uint64_t lanes_below() { return (uint64_t(1) << (threadIdx.x & 63)) - 1; }

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
// their leader with one atomic (scores cluster in a few bins); after four rounds
// the remaining lanes add individually.
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
  }
  if ((act >> lane) & 1u) atomicAdd(&hist[bin], 1u);
}

__global__ void __launch_bounds__(SEL_THREADS) k_select(const ikv_session *__restrict__ sess,
                                                        const int32_t *__restrict__ slot_maps, int dead,
                                                        const float *__restrict__ scores, uint8_t *__restrict__ keep,
                                                        int32_t *__restrict__ n_keep, float *__restrict__ tau) {
  __shared__ uint32_t keys[SEL_LDS_KEYS];
  __shared__ uint32_t hist[SEL_BINS];
  __shared__ int red[SEL_WAVES];
  __shared__ uint32_t sh_prefix;
  __shared__ int sh_k;
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x, lane = t & 63;
  const int32_t *S = slot_maps + s.slot_off;
  const float *sc = scores + s.slot_off;
  uint8_t *kp = keep + s.slot_off;
  const bool cached = s.N <= SEL_LDS_KEYS;
  auto forced_at = [&](int j) { return j < s.pi || (j >= s.qs && j < s.qe); };
  // slot and score of position j (past the end: a dead position)
  auto load = [&](int j, int &sv, float &fv, bool need_score) {
    sv = j < s.N ? S[j] : dead;
    fv = (need_score && j < s.N) ? sc[j] : 0.f;
  };
  // key of a live candidate, 0 otherwise
  auto key_of = [&](int j, int sv, float fv) -> uint32_t {
    if (j >= s.N) return 0u;
    if (cached) return keys[j];
    return (sv != dead && !forced_at(j)) ? score_key(fv) : 0u;
  };

  // counts of live and forced positions; the candidates' keys go to LDS
  int nl = 0, nf = 0;
  for (int c0 = 0; c0 < s.N; c0 += SEL_THREADS * SEL_U) {
    int sv[SEL_U];
    float fv[SEL_U];
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) load(c0 + u * SEL_THREADS + t, sv[u], fv[u], cached);
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) {
      const int j = c0 + u * SEL_THREADS + t;
      if (j >= s.N) continue;
      const bool live = sv[u] != dead;
      const bool forced = forced_at(j);
      nl += live;
      nf += live && forced;
      if (cached) keys[j] = (live && !forced && s.N > s.C) ? score_key(fv[u]) : 0u;
    }
  }
  nl = block_sum(nl, red);
  nf = block_sum(nf, red);
  const int na = nl - nf;

  if (s.N <= s.C) {   // the compression event is skipped: every live position stays
    for (int j = t; j < s.N; j += SEL_THREADS) kp[j] = S[j] != dead;
    if (t == 0) {
      n_keep[b] = nl;
      tau[b] = -INFINITY;
    }
    return;
  }
  const int cstar = max(0, s.C - nf);
  const int take = min(cstar, na);

  // radix select of the take-th largest key: 11, 11 and 10 bits from the top
  uint32_t prefix = 0;
  int kk = take;
  if (take > 0) {
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
      const uint32_t nbins = pass == 2 ? 1024u : 2048u;
      const uint32_t himask = pass == 0 ? 0u : (0xffffffffu << (shift + (pass == 1 ? 11 : 10)));
      for (int i = t; i < SEL_BINS; i += SEL_THREADS) hist[i] = 0;
      __syncthreads();
      for (int c0 = 0; c0 < s.N; c0 += SEL_THREADS * SEL_U) {
        int sv[SEL_U];
        float fv[SEL_U];
        if (!cached)
#pragma unroll
          for (int u = 0; u < SEL_U; ++u) load(c0 + u * SEL_THREADS + t, sv[u], fv[u], true);
#pragma unroll
        for (int u = 0; u < SEL_U; ++u) {
          const int j = c0 + u * SEL_THREADS + t;
          const uint32_t key = key_of(j, sv[u], fv[u]);
          const bool on = key != 0u && (key & himask) == (prefix & himask);
          hist_add(hist, (key >> shift) & (nbins - 1u), on);
        }
      }
      __syncthreads();
      // thread t owns bins 2t, 2t+1 (pass 2: bin t); find the bin holding the kk-th
      // largest by an exclusive scan over threads from the top bin down
      const int per = pass == 2 ? 1 : 2;
      const int hi_bin = int(nbins) - 1 - t * per;        // highest bin of this thread
      int c = 0;
      if (hi_bin >= 0)
        for (int q = 0; q < per; ++q) c += int(hist[hi_bin - q]);
      int x = c;                                          // inclusive scan in thread order
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, WAVE);
        if (lane >= o) x += y;
      }
      int tot;
      const int wb = wave_base(__shfl(x, 63, WAVE), tot, red);
      const int above = wb + x - c;                       // keys in bins above this thread's
      if (hi_bin >= 0 && above < kk && kk <= above + c) {
        int cum = above;
        for (int q = 0; q < per; ++q) {
          const int bin = hi_bin - q;
          const int h = int(hist[bin]);
          if (cum + h >= kk) {
            sh_prefix = prefix | (uint32_t(bin) << shift);
            sh_k = kk - cum;
            break;
          }
          cum += h;
        }
      }
      __syncthreads();
      prefix = sh_prefix;
      kk = sh_k;
      __syncthreads();
    }
  }

  // keep F, every candidate above the threshold key, and the first kk equal to it in
  // position order: wave w ranks the ties of its own contiguous range
  int64_t lo, hi;
  wave_range(s.N, lo, hi);
  int ties = 0;
  if (take > 0)
    for (int64_t c0 = lo; c0 < hi; c0 += WAVE * SEL_U) {
      int sv[SEL_U];
      float fv[SEL_U];
      if (!cached)
#pragma unroll
        for (int u = 0; u < SEL_U; ++u) load(int(c0) + u * WAVE + lane, sv[u], fv[u], true);
#pragma unroll
      for (int u = 0; u < SEL_U; ++u) {
        const int j = int(c0) + u * WAVE + lane;
        const bool eq = j < hi && key_of(j, sv[u], fv[u]) == prefix;
        ties += __popcll(__ballot(eq));
      }
    }
  int all_ties;
  int rank = wave_base(ties, all_ties, red);
  int kept = 0;
  for (int64_t c0 = lo; c0 < hi; c0 += WAVE * SEL_U) {
    int sv[SEL_U];
    float fv[SEL_U];
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) load(int(c0) + u * WAVE + lane, sv[u], fv[u], !cached);
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) {
      const int j = int(c0) + u * WAVE + lane;
      bool k = false, eq = false;
      if (j < hi) {
        const bool live = sv[u] != dead;
        if (live && forced_at(j)) {
          k = true;
        } else if (live && take > 0) {
          const uint32_t key = key_of(j, sv[u], fv[u]);
          k = key > prefix;
          eq = key == prefix;
        }
      }
      const uint64_t bal = __ballot(eq);
      if (eq && rank + __popcll(bal & lanes_below()) < kk) k = true;
      rank += __popcll(bal);
      if (j < hi) kp[j] = k ? 1 : 0;
      kept += k;
    }
  }
  kept = block_sum(kept, red);
  if (t == 0) {
    n_keep[b] = kept;
    tau[b] = take > 0 ? key_score(prefix) : INFINITY;
  }
}

hipError_t launch_select(const ikv_session *sess_dev, int B, int, const int32_t *slot_maps, int32_t dead,
                         const float *scores, uint8_t *keep, int32_t *n_keep, float *tau, hipStream_t st) {
  {
    KTimer kt_("k_select", st);
    k_select<<<B, SEL_THREADS, 0, st>>>(sess_dev, slot_maps, dead, scores, keep, n_keep, tau);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ redirect
// The two slot bitsets (slots of kept positions, freed slots) live in LDS when the
// pool has at most RED_LDS_WORDS * 32 slots, else in the caller's workspace, where
// the workgroup's waves reach each other through device-scope atomics and fences.
constexpr int RED_LDS_WORDS = 16384;        // two bitsets of 64 KB: pools up to 524288 slots

template <bool LDS_SETS>
struct SlotSets {
  uint32_t *kept, *freed;
  __device__ __forceinline__ void set(uint32_t *w, int u) const {
    if (LDS_SETS) atomicOr(w + (u >> 5), 1u << (u & 31));
    else __hip_atomic_fetch_or(w + (u >> 5), 1u << (u & 31), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __device__ __forceinline__ uint32_t word(const uint32_t *w, int64_t i) const {
    if (LDS_SETS) return w[i];
    return __hip_atomic_load(w + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __device__ __forceinline__ void clear(uint32_t *w, int64_t i) const {
    if (LDS_SETS) w[i] = 0u;
    else __hip_atomic_store(w + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __device__ __forceinline__ void sync() const {
    if (!LDS_SETS) __threadfence();
    __syncthreads();
  }
};

template <bool LDS_SETS>
__global__ void __launch_bounds__(SEL_THREADS) k_redirect(const ikv_session *__restrict__ sess, int64_t num_slots,
                                                          int32_t *__restrict__ slot_maps, int dead,
                                                          const uint8_t *__restrict__ keep, int32_t *__restrict__ freed,
                                                          int32_t *__restrict__ n_freed, int32_t *__restrict__ live,
                                                          int32_t *__restrict__ n_live, uint32_t *__restrict__ ws) {
  __shared__ uint32_t lds_sets[LDS_SETS ? 2 * RED_LDS_WORDS : 1];
  __shared__ int red[SEL_WAVES];
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x, lane = t & 63;
  int32_t *S = slot_maps + s.slot_off;
  const uint8_t *kp = keep + s.slot_off;
  const int64_t words = bitset_words(num_slots);
  SlotSets<LDS_SETS> sets;
  sets.kept = LDS_SETS ? lds_sets : ws + int64_t(b) * 2 * words;
  sets.freed = sets.kept + words;

  for (int64_t i = t; i < words; i += SEL_THREADS) {
    sets.clear(sets.kept, i);
    sets.clear(sets.freed, i);
  }
  sets.sync();
  // slots of the kept positions, and the survivors of each wave's range
  int64_t lo, hi;
  wave_range(s.N, lo, hi);
  int surv = 0;
  for (int64_t c0 = lo; c0 < hi; c0 += WAVE * SEL_U) {
    int sv[SEL_U];
    uint8_t kv[SEL_U];
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) {
      const int j = int(c0) + u * WAVE + lane;
      sv[u] = j < hi ? S[j] : dead;
      kv[u] = j < hi ? kp[j] : 0;
    }
#pragma unroll
    for (int u = 0; u < SEL_U; ++u) {
      const bool k = sv[u] != dead && kv[u] != 0;
      if (k) sets.set(sets.kept, sv[u]);
      surv += __popcll(__ballot(k));
    }
  }
  int total_live;
  int pos = wave_base(surv, total_live, red);
  sets.sync();
  // reroute dropped positions, mark freeable slots, list the survivors in position order
  for (int64_t c0 = lo; c0 < hi; c0 += WAVE * SEL_U) {
    int sv[SEL_U];
    uint8_t kv[SEL_U];
#pragma unroll
    for (int q = 0; q < SEL_U; ++q) {
      const int j = int(c0) + q * WAVE + lane;
      sv[q] = j < hi ? S[j] : dead;
      kv[q] = j < hi ? kp[j] : 0;
    }
#pragma unroll
    for (int q = 0; q < SEL_U; ++q) {
      const int j = int(c0) + q * WAVE + lane;
      const int u = sv[q];
      const bool alive = u != dead;
      const bool k = alive && kv[q] != 0;
      if (alive && !k) {
        S[j] = dead;
        if (j >= s.radix_prefix && !((sets.word(sets.kept, u >> 5) >> (u & 31)) & 1u)) sets.set(sets.freed, u);
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
  for (int64_t c0 = wlo; c0 < whi; c0 += WAVE) {
    const int64_t i = c0 + lane;
    const uint32_t bits = i < whi ? sets.word(sets.freed, i) : 0u;
    const int c = __popc(bits);
    int x = c;                                      // inclusive scan over the lanes
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, WAVE);
      if (lane >= o) x += y;
    }
    int r = fpos + x - c;
    uint32_t m = bits;
    while (m) {
      const int bit = __ffs(m) - 1;
      m &= m - 1;
      freed[s.slot_off + r] = int32_t(i * 32 + bit);
      ++r;
    }
    fpos += __shfl(x, 63, WAVE);
  }
  if (t == 0) n_freed[b] = total_freed;
}

hipError_t launch_redirect(const ikv_session *sess_dev, int B, int64_t num_slots, int32_t *slot_maps, int32_t dead,
                           const uint8_t *keep, int32_t *freed, int32_t *n_freed, int32_t *live, int32_t *n_live,
                           uint32_t *ws, hipStream_t st) {
  if (bitset_words(num_slots) <= RED_LDS_WORDS)
    {
      KTimer kt_("k_redirect<true>", st);
      k_redirect<true><<<B, SEL_THREADS, 0, st>>>(sess_dev, num_slots, slot_maps, dead, keep, freed, n_freed, live,
                                                  n_live, ws);
    }
  else
    {
      KTimer kt_("k_redirect<false>", st);
      k_redirect<false><<<B, SEL_THREADS, 0, st>>>(sess_dev, num_slots, slot_maps, dead, keep, freed, n_freed, live,
                                                   n_live, ws);
    }
  return hipGetLastError();
}

}  // namespace ikv
