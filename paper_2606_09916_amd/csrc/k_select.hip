// Budgeted selection of Eq. 1 (Appendix H: K = F u topk(A, max(0, C - |F|))) and
// the slot-map redirect of Eq. 7 with the alias-aware free of Sec. 3.4.
//
// Both run one 1024-thread workgroup per session: a session's positions are a
// few hundred KB at most, and every step here is integer work or a comparison.
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_WAVES = SEL_THREADS / WAVE;

// Exclusive prefix sum over the workgroup in thread order; `total` gets the sum.
// `lds` holds SEL_WAVES + 1 ints. Every thread of the workgroup must call it.
__device__ __forceinline__ int block_excl_scan(int v, int &total, int *lds) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, WAVE);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int w = 0; w < SEL_WAVES; ++w) {
      const int c = lds[w];
      lds[w] = acc;
      acc += c;
    }
    lds[SEL_WAVES] = acc;
  }
  __syncthreads();
  const int r = lds[wave] + x - v;
  total = lds[SEL_WAVES];
  __syncthreads();
  return r;
}

__device__ __forceinline__ int block_sum(int v, int *lds) {
  int total;
  block_excl_scan(v, total, lds);
  return total;
}

// Order-preserving map of a score to an unsigned key: larger score, larger key.
// NaN is ranked as -inf and -0.0 as +0.0.
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

__global__ void __launch_bounds__(SEL_THREADS) k_select(const ikv_session *__restrict__ sess,
                                                        const int32_t *__restrict__ slot_maps, int dead,
                                                        const float *__restrict__ scores, uint8_t *__restrict__ keep,
                                                        int32_t *__restrict__ n_keep, float *__restrict__ tau) {
  __shared__ int lds[SEL_WAVES + 1];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_prefix;
  __shared__ int sh_k;
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x;
  const int32_t *S = slot_maps + s.slot_off;
  const float *sc = scores + s.slot_off;
  uint8_t *kp = keep + s.slot_off;

  // counts of live, forced and candidate positions
  int nl = 0, nf = 0;
  for (int j = t; j < s.N; j += SEL_THREADS) {
    const bool live = S[j] != dead;
    const bool forced = j < s.pi || (j >= s.qs && j < s.qe);
    nl += live;
    nf += live && forced;
  }
  nl = block_sum(nl, lds);
  nf = block_sum(nf, lds);
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

  // radix select of the take-th largest key, 8 bits per pass from the top
  uint32_t prefix = 0;
  int kk = take;
  if (take > 0) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      const uint32_t himask = pass == 0 ? 0u : (0xffffffffu << (32 - 8 * pass));
      for (int i = t; i < 256; i += SEL_THREADS) hist[i] = 0;
      __syncthreads();
      for (int j = t; j < s.N; j += SEL_THREADS) {
        if (S[j] == dead || j < s.pi || (j >= s.qs && j < s.qe)) continue;
        const uint32_t key = score_key(sc[j]);
        if ((key & himask) == (prefix & himask)) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (t == 0) {
        int cum = 0;
        for (int bin = 255; bin >= 0; --bin) {
          const int c = int(hist[bin]);
          if (cum + c >= kk) {
            sh_prefix = prefix | (uint32_t(bin) << shift);
            sh_k = kk - cum;
            break;
          }
          cum += c;
        }
      }
      __syncthreads();
      prefix = sh_prefix;
      kk = sh_k;
      __syncthreads();
    }
  }
  // keep F, every candidate above the threshold key, and the first kk equal to it
  int base = 0, kept = 0;
  for (int c0 = 0; c0 < s.N; c0 += SEL_THREADS) {
    const int j = c0 + t;
    bool k = false, eq = false;
    if (j < s.N) {
      const bool live = S[j] != dead;
      const bool forced = j < s.pi || (j >= s.qs && j < s.qe);
      if (live && forced) {
        k = true;
      } else if (live && take > 0) {
        const uint32_t key = score_key(sc[j]);
        k = key > prefix;
        eq = key == prefix;
      }
    }
    int tot;
    const int r = block_excl_scan(eq ? 1 : 0, tot, lds);
    if (eq && base + r < kk) k = true;
    base += tot;
    if (j < s.N) kp[j] = k ? 1 : 0;
    kept += k;
  }
  kept = block_sum(kept, lds);
  if (t == 0) {
    n_keep[b] = kept;
    tau[b] = take > 0 ? key_score(prefix) : INFINITY;
  }
}

hipError_t launch_select(const ikv_session *sess_dev, int B, int, const int32_t *slot_maps, int32_t dead,
                         const float *scores, uint8_t *keep, int32_t *n_keep, float *tau, hipStream_t st) {
  k_select<<<B, SEL_THREADS, 0, st>>>(sess_dev, slot_maps, dead, scores, keep, n_keep, tau);
  return hipGetLastError();
}

// ------------------------------------------------------------------ redirect
__device__ __forceinline__ uint32_t load_coherent(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void __launch_bounds__(SEL_THREADS) k_redirect(const ikv_session *__restrict__ sess, int64_t num_slots,
                                                          int32_t *__restrict__ slot_maps, int dead,
                                                          const uint8_t *__restrict__ keep, int32_t *__restrict__ freed,
                                                          int32_t *__restrict__ n_freed, int32_t *__restrict__ live,
                                                          int32_t *__restrict__ n_live, uint32_t *__restrict__ ws) {
  __shared__ int lds[SEL_WAVES + 1];
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x;
  int32_t *S = slot_maps + s.slot_off;
  const uint8_t *kp = keep + s.slot_off;
  const int64_t words = bitset_words(num_slots);
  uint32_t *kept_set = ws + int64_t(b) * 2 * words;
  uint32_t *free_set = kept_set + words;

  for (int64_t i = t; i < words; i += SEL_THREADS) {
    __hip_atomic_store(kept_set + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(free_set + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __threadfence();
  __syncthreads();
  // slots of the kept positions
  for (int j = t; j < s.N; j += SEL_THREADS) {
    const int u = S[j];
    if (u != dead && kp[j]) atomicOr(kept_set + (u >> 5), 1u << (u & 31));
  }
  __threadfence();
  __syncthreads();
  // reroute dropped positions, mark freeable slots, list the survivors in position order
  int base = 0;
  for (int c0 = 0; c0 < s.N; c0 += SEL_THREADS) {
    const int j = c0 + t;
    int u = dead;
    bool k = false;
    if (j < s.N) {
      u = S[j];
      k = kp[j] != 0;
    }
    const bool alive = u != dead;
    if (alive && !k) {
      S[j] = dead;
      if (j >= s.radix_prefix && !((load_coherent(kept_set + (u >> 5)) >> (u & 31)) & 1u))
        atomicOr(free_set + (u >> 5), 1u << (u & 31));
    }
    int tot;
    const int r = block_excl_scan(alive && k ? 1 : 0, tot, lds);
    if (alive && k) live[s.slot_off + base + r] = u;
    base += tot;
  }
  __threadfence();
  __syncthreads();
  if (t == 0) n_live[b] = base;
  // freed slots in ascending slot order
  int fbase = 0;
  for (int64_t w0 = 0; w0 < words; w0 += SEL_THREADS) {
    const int64_t w = w0 + t;
    const uint32_t bits = w < words ? load_coherent(free_set + w) : 0u;
    int tot;
    int r = block_excl_scan(__popc(bits), tot, lds);
    uint32_t m = bits;
    while (m) {
      const int bit = __ffs(m) - 1;
      m &= m - 1;
      freed[s.slot_off + fbase + r] = int32_t(w * 32 + bit);
      ++r;
    }
    fbase += tot;
  }
  if (t == 0) n_freed[b] = fbase;
}

hipError_t launch_redirect(const ikv_session *sess_dev, int B, int64_t num_slots, int32_t *slot_maps, int32_t dead,
                           const uint8_t *keep, int32_t *freed, int32_t *n_freed, int32_t *live, int32_t *n_live,
                           uint32_t *ws, hipStream_t st) {
  k_redirect<<<B, SEL_THREADS, 0, st>>>(sess_dev, num_slots, slot_maps, dead, keep, freed, n_freed, live, n_live,
                                        ws);
  return hipGetLastError();
}

}  // namespace ikv
