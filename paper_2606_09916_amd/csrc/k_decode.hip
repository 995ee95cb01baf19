// GQA decode attention over the live slots of each session (the kept entries read
// through the slot map with the sentinel stripped, Sec. 3.4 and Appendix C.2).
//
// Two kernels write the partial state of each split: k_decode_heads (bf16 pool,
// D = 128; logits on the matrix cores, described where it is defined) and
// k_decode_split (every other pool), below.
//
// k_decode_split: one workgroup per (session, layer, KV head, split of the live
// list). Each wavefront takes blocks of 64 live slots: lane k computes the logits
// of slot k for the G query heads sharing the KV head, the block's weights are
// folded into a running (max, sum, output) per head. The value rows only need the
// slots, so they are loaded together with the key rows (16 bytes per lane, 64 / (D/8)
// rows per load instruction); the lanes of one channel group fold their rows at the end.
// The partial state of every split goes to the workspace, the output rows of all
// splits first ([part][D], each row 512 aligned bytes at D = 128, written as whole
// 16-byte pieces) and their (max, sum) pairs after them ([part][2]); k_decode_combine
// merges the splits per (session, layer, head).
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

// Workgroups per (session, layer) of the decode kernel for this pool: one per group of
// adjacent KV heads in the head-group kernel, one per KV head otherwise.
int64_t decode_units(const ikv_pool &p, int B) {
  if (p.kv_dtype == IKV_BF16 && p.D == 128) {
    const int hpw = p.Hkv % 4 == 0 ? 4 : (p.Hkv % 2 == 0 ? 2 : 1);
    return int64_t(B) * p.L * (p.Hkv / hpw);
  }
  return int64_t(B) * p.L * p.Hkv;
}

// Splits of the live list: enough workgroups for about one resident round (two per CU
// on the 256 CUs of MI355X), at least 64 live positions per split, at most 64 splits.
// A workgroup ends with its split's stores, and its slot takes no new work until they
// are done; long splits in one round pay that once per slot. At the Qwen3-8B 32k step
// (8192 live, 72 units) that is 7 splits of 1171 positions: the head-group kernel
// 196 us against 212 with 32 splits of 256 (without the stores, 32 splits ran in 191).
int decode_splits(int live_bound, int64_t units) {
  int64_t s = 512 / (units < 1 ? 1 : units);
  s = std::min<int64_t>(s, cdiv(live_bound, 64));
  return int(s < 1 ? 1 : (s > 64 ? 64 : s));
}

// 8 consecutive elements kept as raw 16-byte words until they are used.
template <typename T> struct Raw8 {
  static constexpr int W = sizeof(T) / 2;      // uint4 words: 1 for bf16, 2 for float
  uint4 r[W];
  __device__ __forceinline__ void ld(const T *p) {
#pragma unroll
    for (int k = 0; k < W; ++k) r[k] = reinterpret_cast<const uint4 *>(p)[k];
  }
  __device__ __forceinline__ void unpack(float (&o)[8]) const {
    if constexpr (W == 1) {
      const uint32_t w[4] = {r[0].x, r[0].y, r[0].z, r[0].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        o[2 * i] = __uint_as_float(w[i] << 16);
        o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
      }
    } else {
      const uint32_t w[8] = {r[0].x, r[0].y, r[0].z, r[0].w, r[1].x, r[1].y, r[1].z, r[1].w};
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = __uint_as_float(w[i]);
    }
  }
};

// The end of a split: fold the value row groups of each wavefront, merge the four
// wavefronts through LDS, and write (max, sum, output) per query head to the workspace.
template <int D, int G>
__device__ __forceinline__ void decode_finish(float (&m)[G], float (&lsum)[G], float (&o)[G][8], float (&red)[4][G][2],
                                              float (&ored)[4][G][D], float *__restrict__ ws, float *__restrict__ ws_ml,
                                              int b, int L, int l, int Hq, int g, int split, int nsplit) {
  constexpr int LPR = D / 8;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int rq = lane / LPR, cq = lane % LPR;
  // fold the value row groups of each wavefront, then merge the four wavefronts
#pragma unroll
  for (int x = LPR; x < WAVE; x <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int c = 0; c < 8; ++c) o[h][c] += __shfl_xor(o[h][c], x, WAVE);
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      red[w][h][0] = m[h];
      red[w][h][1] = lsum[h];
    }
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float mm = -INFINITY;
    for (int k = 0; k < 4; ++k) mm = fmaxf(mm, red[k][h][0]);
    const float f = (m[h] == -INFINITY) ? 0.f : __expf(m[h] - mm);
    if (rq == 0)
#pragma unroll
      for (int c = 0; c < 8; ++c) ored[w][h][cq * 8 + c] = o[h][c] * f;
  }
  __syncthreads();
  for (int e = t; e < G * (D + 2); e += 256) {
    const int h = e / (D + 2), d = e - h * (D + 2);
    const int64_t part = ((int64_t(b) * L + l) * Hq + g * G + h) * nsplit + split;
    float mm = -INFINITY;
    for (int k = 0; k < 4; ++k) mm = fmaxf(mm, red[k][h][0]);
    if (d == 0) {
      ws_ml[part * 2] = mm;
    } else if (d == 1) {
      float val = 0.f;
      for (int k = 0; k < 4; ++k)
        if (red[k][h][0] != -INFINITY) val += red[k][h][1] * __expf(red[k][h][0] - mm);
      ws_ml[part * 2 + 1] = val;
    } else {
      ws[part * D + d - 2] = (ored[0][h][d - 2] + ored[1][h][d - 2]) + (ored[2][h][d - 2] + ored[3][h][d - 2]);
    }
  }
}

template <typename T, int D, int G>
__global__ void __launch_bounds__(256) k_decode_split(const T *__restrict__ kpool, const T *__restrict__ vpool,
                                                      int64_t num_slots, int L, int Hkv,
                                                      const ikv_session *__restrict__ sess, const T *__restrict__ q,
                                                      const int32_t *__restrict__ live,
                                                      const int32_t *__restrict__ n_live, float *__restrict__ ws,
                                                      float *__restrict__ ws_ml) {
  constexpr int LPR = D / 8;           // lanes per value row (8 channels each)
  constexpr int RPI = WAVE / LPR;      // value rows per load instruction
  __shared__ float qs[G][D];
  __shared__ float pw[4][G][DEC_BLOCK];
  __shared__ float red[4][G][2];
  __shared__ float ored[4][G][D];

  const int b = blockIdx.z;
  const ikv_session s = sess[b];
  const int Hq = Hkv * G;
  const int u = blockIdx.y, l = u / Hkv, g = u - l * Hkv;
  const int split = blockIdx.x, nsplit = gridDim.x;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  int n = n_live[b];
  n = n < 0 ? 0 : (n > s.N ? s.N : n);
  const int chunk = int(cdiv(n, nsplit));
  const int k0 = min(n, split * chunk), k1 = min(n, k0 + chunk);
  const float scale = 1.0f / sqrtf(float(D));
  const int32_t *lv = live + s.slot_off;
  int slot0 = 0;                                   // the first block's slot: loads with the query rows
  if (k0 + w * DEC_BLOCK + lane < k1) slot0 = lv[k0 + w * DEC_BLOCK + lane];
  for (int e = t; e < G * D; e += 256) {
    const int h = e / D, d = e - h * D;
    qs[h][d] = Store<T>::ld(q + ((int64_t(b) * L + l) * Hq + g * G + h) * D + d) * scale;
  }
  __syncthreads();
  const int rq = lane / LPR, cq = lane % LPR;     // value row group, channel group
  float m[G], lsum[G], o[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    lsum[h] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[h][i] = 0.f;
  }
  const int64_t row_stride = int64_t(Hkv) * D;
  const T *kbase = kpool + int64_t(l) * num_slots * row_stride + int64_t(g) * D;
  const T *vbase = vpool + int64_t(l) * num_slots * row_stride + int64_t(g) * D;
  for (int base = k0 + w * DEC_BLOCK; base < k1; base += 4 * DEC_BLOCK) {
    const int kk = base + lane;
    const bool valid = kk < k1;
    const int slot = base == k0 + w * DEC_BLOCK ? slot0 : (valid ? lv[kk] : 0);
    const int nb = min(DEC_BLOCK, k1 - base);
    Raw8<T> v[DEC_BLOCK / RPI];
#pragma unroll
    for (int r = 0; r < DEC_BLOCK / RPI; ++r) {
      const int i = r * RPI + rq;
      const int si = __shfl(slot, i, WAVE);
      if (i < nb) v[r].ld(vbase + int64_t(si) * row_stride + cq * 8);
    }
    float x[G];
#pragma unroll
    for (int h = 0; h < G; ++h) x[h] = 0.f;
    if (valid) {
      const T *kr = kbase + int64_t(slot) * row_stride;
      Raw8<T> kraw[D / 8];
#pragma unroll
      for (int d = 0; d < D; d += 8) kraw[d / 8].ld(kr + d);
#pragma unroll
      for (int d = 0; d < D; d += 8) {
        float kv[8];
        kraw[d / 8].unpack(kv);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float4 q0 = *reinterpret_cast<const float4 *>(&qs[h][d]);
          const float4 q1 = *reinterpret_cast<const float4 *>(&qs[h][d + 4]);
          x[h] = fmaf(kv[0], q0.x, x[h]);
          x[h] = fmaf(kv[1], q0.y, x[h]);
          x[h] = fmaf(kv[2], q0.z, x[h]);
          x[h] = fmaf(kv[3], q0.w, x[h]);
          x[h] = fmaf(kv[4], q1.x, x[h]);
          x[h] = fmaf(kv[5], q1.y, x[h]);
          x[h] = fmaf(kv[6], q1.z, x[h]);
          x[h] = fmaf(kv[7], q1.w, x[h]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float xv = valid ? x[h] : -INFINITY;
      const float mn = fmaxf(m[h], wave_max(xv));
      const float corr = (m[h] == -INFINITY) ? 0.f : __expf(m[h] - mn);
      const float p = valid ? __expf(xv - mn) : 0.f;
      lsum[h] = lsum[h] * corr + wave_sum(p);
      m[h] = mn;
      pw[w][h][lane] = p;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[h][i] *= corr;
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
    for (int r = 0; r < DEC_BLOCK / RPI; ++r) {
      const int i = r * RPI + rq;
      if (i < nb) {
        float vv[8];
        v[r].unpack(vv);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = pw[w][h][i];
#pragma unroll
          for (int c = 0; c < 8; ++c) o[h][c] = fmaf(p, vv[c], o[h][c]);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  }
  decode_finish<D, G>(m, lsum, o, red, ored, ws, ws_ml, b, L, l, Hq, g, split, nsplit);
}

typedef __bf16 bf16x8_d __attribute__((ext_vector_type(8)));
typedef float f32x4_d __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_d __attribute__((ext_vector_type(4)));

// ---- head-group decode (bf16 pool, D = 128). A workgroup owns a group of `hpw`
// adjacent KV heads of one layer (hpw * 256 contiguous bytes of every key and value
// row) and one split of the live list; wave w owns KV head g0 + w and walks the whole
// split in halves of 32 live slots (16 for G > 4), so the waves of a workgroup read
// adjacent pieces of the same rows together. The value rows have two register buffers,
// the key fragments one: at the top of each half the next half's value rows are
// issued, then the current half's logits run on the matrix cores, then the next half's
// key fragments are issued into the registers those MFMAs have read, and the softmax
// update and weighted value sums finish the half. Every path issues the same loads in
// the same order (rows past the end of the split read the split's first live row and
// get weight zero; the next pair's slot list is loaded at the top of the current pair,
// its index clamped), so the compiler's memory waits are exact counts and no half
// waits for loads issued after its own. Each wave writes its own (max, sum, output)
// per query head.
// The value rows load with the non-temporal hint (each instruction reads 4 whole
// 256-byte rows); the key loads keep the default policy (each instruction reads one
// 64-byte quarter of 16 rows, and the next instructions read the rest of the same lines).
template <int G, bool O32>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) k_decode_heads(const uint16_t *__restrict__ kpool,
                                                      const uint16_t *__restrict__ vpool, int64_t num_slots, int L,
                                                      int Hkv, int hpw, const ikv_session *__restrict__ sess,
                                                      const uint16_t *__restrict__ q, const int32_t *__restrict__ live,
                                                      const int32_t *__restrict__ n_live, float *__restrict__ ws,
                                                      float *__restrict__ ws_ml) {
  constexpr int D = 128;
  constexpr int HB = G <= 4 ? 32 : 16; // live slots per half (fewer where the G output rows take the registers)
  constexpr int LPR = D / 8;           // lanes per value row (8 channels each)
  constexpr int RPI = WAVE / LPR;      // value rows per load instruction
  constexpr int NV = HB / RPI;         // value loads per half
  constexpr int NB = HB / 16;          // 16-row MFMA blocks per half
  constexpr int GP = (G + 3) & ~3;     // weights per position in LDS, padded to float4
  __shared__ __align__(16) float pw[4][HB][GP];
  __shared__ __align__(16) bf16x8_d qsh[4][4][WAVE];   // query fragments, read before every half's MFMAs

  const int b = blockIdx.z;
  const ikv_session s = sess[b];
  const int Hq = Hkv * G;
  const int ngrp = Hkv / hpw;
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int l = blockIdx.y / ngrp, g = (blockIdx.y - l * ngrp) * hpw + w;
  const int split = blockIdx.x, nsplit = gridDim.x;
  const int gq = lane >> 4, r16 = lane & 15;
  const int rq = lane / LPR, cq = lane % LPR;     // value row group, channel group
  int n = n_live[b];
  n = n < 0 ? 0 : (n > s.N ? s.N : n);
  const int chunk = int(cdiv(n, nsplit));          // the halves take any length, so splits differ by one at most
  const int k0 = min(n, split * chunk), k1 = min(n, k0 + chunk);
  const float scale = 1.0f / sqrtf(float(D));
  const int32_t *lv = live + s.slot_off;
  // the query rows as the B operand: lane (gq, r16) holds channels ks*32 + gq*8 .. +8 of head r16.
  // They stay in LDS (no registers to spare beside two halves of key and value loads).
  {
    const uint16_t *qr = q + ((int64_t(b) * L + l) * Hq + g * G + (r16 < G ? r16 : 0)) * D + gq * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      bf16x8_d x = *reinterpret_cast<const bf16x8_d *>(qr + ks * 32);
      if (r16 >= G) x = bf16x8_d{};
      qsh[w][ks][lane] = x;
    }
  }
  float m[G], lsum[G], o[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    lsum[h] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[h][i] = 0.f;
  }
  if (k0 < k1) {
    const int64_t row_stride = int64_t(Hkv) * D;
    // wave-uniform bases (this wave's head in layer l); a row is reached by a per-lane
    // byte offset, 32 bits wide when a layer of the pool spans less than 4 GB
    const char *kbase = reinterpret_cast<const char *>(kpool + int64_t(l) * num_slots * row_stride + int64_t(g) * D);
    const char *vbase = reinterpret_cast<const char *>(vpool + int64_t(l) * num_slots * row_stride + int64_t(g) * D);
    const uint32_t row_bytes = uint32_t(row_stride) * 2;
    auto row_off = [&](int sl, int within) -> uint64_t {
      if constexpr (O32) return uint32_t(sl) * row_bytes + uint32_t(within);
      else return uint64_t(uint32_t(sl)) * row_bytes + uint32_t(within);
    };
    // slots of the pair starting at `base`, one per lane: past the split's end the
    // split's first live slot (its row is read again and weighted zero); the index is
    // clamped, so the load is the same on every path
    const int first = lv[k0];
    auto pair_slots = [&](int base) {
      const int i = base + lane;
      const int sl = lv[min(i, k1 - 1)];
      return i < k1 ? sl : first;
    };
    Raw8<uint16_t> va[NV], vb[NV];
    bf16x8_d kf[NB][4];
    // slot of lane j of `sl` for the key rows (j = off + 16 bb + r16) and the value rows
    // (j = off + 4 r + rq): one byte address per lane, the rest an immediate offset
    const int kaddr = r16 * 4, vaddr = rq * 4;
    auto pick = [](int addr, int sl) { return __builtin_amdgcn_ds_bpermute(addr, sl); };
    // the key fragments (into kf) and the value rows (into v) of the half at lane offset
    // `off` of a pair
    auto load_k = [&](int sl, int off) __attribute__((always_inline)) {
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) {
        const int sr = pick(kaddr + 4 * (off + bb * 16), sl);
        const char *kr = kbase + row_off(sr, gq * 16);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) kf[bb][ks] = *reinterpret_cast<const bf16x8_d *>(kr + ks * 64);
      }
    };
    auto load_v = [&](Raw8<uint16_t> (&v)[NV], int sl, int off) __attribute__((always_inline)) {
#pragma unroll
      for (int r = 0; r < NV; ++r) {
        const int si = pick(vaddr + 4 * (off + r * RPI), sl);
        const u32x4_d x = __builtin_nontemporal_load(reinterpret_cast<const u32x4_d *>(vbase + row_off(si, cq * 16)));
        v[r].r[0] = make_uint4(x.x, x.y, x.z, x.w);
      }
    };
    // the logits of the half in kf: acc[bb][i] is position bb*16 + 4gq + i, query head r16
    f32x4_d acc[NB];
    auto logits = [&]() __attribute__((always_inline)) {
      asm volatile("" ::: "memory");               // re-read the query fragments every half
#pragma unroll
      for (int bb = 0; bb < NB; ++bb) acc[bb] = f32x4_d{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8_d qb = qsh[w][ks][lane];
#pragma unroll
        for (int bb = 0; bb < NB; ++bb)
          acc[bb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[bb][ks], qb, acc[bb], 0, 0, 0);
      }
    };
    // the rest of a half of nb (<= HB, may be <= 0) live positions: online softmax and
    // the weighted value rows
    auto half = [&](const Raw8<uint16_t> (&v)[NV], int nb) __attribute__((always_inline)) {
      float mx = -INFINITY;
#pragma unroll
      for (int bb = 0; bb < NB; ++bb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float x = (bb * 16 + 4 * gq + i < nb) ? acc[bb][i] * scale : -INFINITY;
          acc[bb][i] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, WAVE));
      mx = fmaxf(mx, __shfl_xor(mx, 32, WAVE));
      float mn[G], corr[G];
#pragma unroll
      for (int h = 0; h < G; ++h) {
        mn[h] = fmaxf(m[h], __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, mx), h)));
        corr[h] = (m[h] == -INFINITY) ? 0.f : __expf(m[h] - mn[h]);
      }
      float mine = mn[0];                          // the new max of this lane's head
#pragma unroll
      for (int h = 1; h < G; ++h) mine = (r16 == h) ? mn[h] : mine;
      float ps = 0.f;
#pragma unroll
      for (int bb = 0; bb < NB; ++bb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = (acc[bb][i] == -INFINITY) ? 0.f : __expf(acc[bb][i] - mine);
          ps += p;
          if (r16 < G) pw[w][bb * 16 + 4 * gq + i][r16] = p;
        }
      ps += __shfl_xor(ps, 16, WAVE);
      ps += __shfl_xor(ps, 32, WAVE);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        lsum[h] = lsum[h] * corr[h] + __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ps), h));
        m[h] = mn[h];
#pragma unroll
        for (int c = 0; c < 8; ++c) o[h][c] *= corr[h];
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
      // rows past nb carry weight zero (their logits were masked to -inf)
#pragma unroll
      for (int r = 0; r < NV; ++r) {
        const int i = r * RPI + rq;
        float vv[8];
        v[r].unpack(vv);
        float pv[GP];
#pragma unroll
        for (int h4 = 0; h4 < GP; h4 += 4) {
          const float4 x = *reinterpret_cast<const float4 *>(&pw[w][i][h4]);
          pv[h4] = x.x;
          pv[h4 + 1] = x.y;
          pv[h4 + 2] = x.z;
          pv[h4 + 3] = x.w;
        }
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
          for (int c = 0; c < 8; ++c) o[h][c] = fmaf(pv[h], vv[c], o[h][c]);
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    };
    // Per half: issue the next half's value rows, run the logits (the MFMAs read kf),
    // issue the next half's key fragments into kf, then finish the half. Past the end of
    // the split the loads read the first live row again and are not used.
    int sl = pair_slots(k0);
    load_v(va, sl, 0);
    load_k(sl, 0);
    for (int base = k0; base < k1; base += 2 * HB) {
      const int nsl = pair_slots(base + 2 * HB);     // the next pair's slots (clamped past the end)
      __builtin_amdgcn_sched_barrier(0);
      load_v(vb, sl, HB);                            // this pair's second half
      __builtin_amdgcn_sched_barrier(0);
      logits();
      __builtin_amdgcn_sched_barrier(0);
      load_k(sl, HB);
      __builtin_amdgcn_sched_barrier(0);
      half(va, k1 - base);
      __builtin_amdgcn_sched_barrier(0);
      load_v(va, nsl, 0);                            // the next pair's first half
      __builtin_amdgcn_sched_barrier(0);
      logits();
      __builtin_amdgcn_sched_barrier(0);
      load_k(nsl, 0);
      __builtin_amdgcn_sched_barrier(0);
      half(vb, k1 - base - HB);
      sl = nsl;
    }
  }
  // fold the value row groups; lanes 0..LPR-1 then hold channels cq*8 .. +8
#pragma unroll
  for (int x = LPR; x < WAVE; x <<= 1)
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int c = 0; c < 8; ++c) o[h][c] += __shfl_xor(o[h][c], x, WAVE);
  if (lane < LPR) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const int64_t part = ((int64_t(b) * L + l) * Hq + g * G + h) * nsplit + split;
      float4 *p = reinterpret_cast<float4 *>(ws + part * D + cq * 8);   // 32 aligned bytes per lane
      p[0] = make_float4(o[h][0], o[h][1], o[h][2], o[h][3]);
      p[1] = make_float4(o[h][4], o[h][5], o[h][6], o[h][7]);
      if (lane == 0) *reinterpret_cast<float2 *>(ws_ml + part * 2) = make_float2(m[h], lsum[h]);
    }
  }
}

// Merge the splits of one (session, layer, query head) in one round trip to memory:
// every thread has its output column of every split in flight while the first
// nsplit lanes load the splits' (max, sum) and share them through LDS; then, with M
// the largest split maximum, out = sum_k o_k e^(m_k - M) / sum_k l_k e^(m_k - M).
// An empty split (m = -inf) weighs zero; a row with no live position gives 0.
template <typename T, int D>
__global__ void __launch_bounds__(D) k_decode_combine(const float *__restrict__ ws, const float *__restrict__ ws_ml,
                                                      int nsplit, int L, int Hq, T *__restrict__ out) {
  constexpr int SMAX = 64;                         // decode_splits() gives at most 64 splits
  constexpr int NW = D / 64;
  __shared__ float sm[SMAX], sl[SMAX], wm[NW];
  const int64_t row = int64_t(blockIdx.y) * L * Hq + blockIdx.x;
  const float *p = ws + row * nsplit * D;
  const int d = threadIdx.x;
  float ok[SMAX];
#pragma unroll
  for (int k = 0; k < SMAX; ++k) ok[k] = k < nsplit ? p[k * D + d] : 0.f;
  float mk = -INFINITY;
  if (d < nsplit) {
    const float2 x = reinterpret_cast<const float2 *>(ws_ml + row * nsplit * 2)[d];
    mk = x.x;
    sm[d] = mk;
    sl[d] = x.y;
  }
  mk = wave_max(mk);
  if ((d & 63) == 0) wm[d >> 6] = mk;
  __syncthreads();
  float M = wm[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) M = fmaxf(M, wm[w]);
  float acc = 0.f, lsum = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int k = 0; k < SMAX; ++k)
      if (k < nsplit && sm[k] != -INFINITY) {
        const float f = expf(sm[k] - M);
        acc = fmaf(ok[k], f, acc);
        lsum = fmaf(sl[k], f, lsum);
      }
  }
  out[row * D + d] = Store<T>::from(lsum > 0.f ? acc / lsum : 0.f);
}

template <typename T, int D, int G>
static hipError_t launch_decode_g(const ikv_pool &p, const ikv_session *sess_dev, int B, int splits, const void *q,
                                  const int32_t *live, const int32_t *n_live, void *out, float *ws, hipStream_t st) {
  // split state: the output rows of every (session, layer, query head, split) first,
  // [part][D], then their (max, sum) pairs, [part][2]
  float *ws_ml = ws + int64_t(B) * p.L * p.Hq * splits * D;
  if constexpr (sizeof(T) == 2 && D == 128) {
    const int hpw = p.Hkv % 4 == 0 ? 4 : (p.Hkv % 2 == 0 ? 2 : 1);
    const dim3 grid(splits, p.L * (p.Hkv / hpw), B);
    KTimer kt_("k_decode_heads<G>", st);
    if (p.num_slots * p.Hkv * D * 2 < (int64_t(1) << 32))
      k_decode_heads<G, true><<<grid, 64 * hpw, 0, st>>>((const uint16_t *)p.k_pool, (const uint16_t *)p.v_pool,
                                                         p.num_slots, p.L, p.Hkv, hpw, sess_dev, (const uint16_t *)q,
                                                         live, n_live, ws, ws_ml);
    else
      k_decode_heads<G, false><<<grid, 64 * hpw, 0, st>>>((const uint16_t *)p.k_pool, (const uint16_t *)p.v_pool,
                                                          p.num_slots, p.L, p.Hkv, hpw, sess_dev, (const uint16_t *)q,
                                                          live, n_live, ws, ws_ml);
  } else {
    KTimer kt_("k_decode_split<T, D, G>", st);
    k_decode_split<T, D, G><<<dim3(splits, p.L * p.Hkv, B), 256, 0, st>>>(
        (const T *)p.k_pool, (const T *)p.v_pool, p.num_slots, p.L, p.Hkv, sess_dev, (const T *)q, live, n_live, ws,
        ws_ml);
  }
  {
    KTimer kt_("k_decode_combine<T, D>", st);
    k_decode_combine<T, D><<<dim3(p.L * p.Hq, B), D, 0, st>>>(ws, ws_ml, splits, p.L, p.Hq, (T *)out);
  }
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_decode_d(const ikv_pool &p, const ikv_session *sd, int B, int splits, const void *q,
                                  const int32_t *live, const int32_t *n_live, void *out, float *ws, hipStream_t st) {
  switch (p.Hq / p.Hkv) {
    case 1: return launch_decode_g<T, D, 1>(p, sd, B, splits, q, live, n_live, out, ws, st);
    case 2: return launch_decode_g<T, D, 2>(p, sd, B, splits, q, live, n_live, out, ws, st);
    case 3: return launch_decode_g<T, D, 3>(p, sd, B, splits, q, live, n_live, out, ws, st);
    case 4: return launch_decode_g<T, D, 4>(p, sd, B, splits, q, live, n_live, out, ws, st);
    case 5: return launch_decode_g<T, D, 5>(p, sd, B, splits, q, live, n_live, out, ws, st);
    case 6: return launch_decode_g<T, D, 6>(p, sd, B, splits, q, live, n_live, out, ws, st);
    case 7: return launch_decode_g<T, D, 7>(p, sd, B, splits, q, live, n_live, out, ws, st);
    default: return launch_decode_g<T, D, 8>(p, sd, B, splits, q, live, n_live, out, ws, st);
  }
}

hipError_t launch_decode(const ikv_pool &p, const ikv_session *sess_dev, int B, int splits, const void *q,
                         const int32_t *live, const int32_t *n_live, void *out, float *ws, hipStream_t st) {
  const bool bf = p.kv_dtype == IKV_BF16;
  if (p.D == 128)
    return bf ? launch_decode_d<uint16_t, 128>(p, sess_dev, B, splits, q, live, n_live, out, ws, st)
              : launch_decode_d<float, 128>(p, sess_dev, B, splits, q, live, n_live, out, ws, st);
  return bf ? launch_decode_d<uint16_t, 64>(p, sess_dev, B, splits, q, live, n_live, out, ws, st)
            : launch_decode_d<float, 64>(p, sess_dev, B, splits, q, live, n_live, out, ws, st);
}

}  // namespace ikv
