// Rule score of Eq. 3 on the matrix cores (bf16 pool, head dimension 128, memory
// rows per KV head a multiple of 16).
//
// The logits x = M . K / sqrt(D) of a unit (layer, KV head) and a tile of 128
// positions form a [128 x R] product with a 128-long contraction. They run as
// v_mfma_f32_16x16x32_bf16 with K (exact in bf16) as the A operand and the memory
// rows as the B operand. Each memory row is pre-split into bf16 hi + lo
// (M' = hi + lo to 2^-18 relative), so two MFMAs per fragment give float32-grade
// logits. log2(e)/sqrt(D) is folded into M', so the softmax uses native exp2.
//
// One workgroup owns 128 positions and walks every unit. The unit's key rows
// stream into a 4-stage LDS ring by direct global->LDS loads (three units in
// flight while one computes); every 16 lanes load one 256-byte row, and the
// row's 16-byte chunks are XOR-swizzled by position so that the MFMA fragment
// reads hit distinct banks. Wave w takes the 16-row slices w, w+4, ... of the
// memory; its first slice's fragments are prefetched one unit ahead.
//   pass A: per (tile, unit, row) the max and sum of exp2 over the tile's candidates;
//   lse:    per (unit, row) the tiles combine into (max, 1/Z);
//   pass B: p = exp2(x - max) / Z summed over every unit and row, per position, in
//           registers; with the residual head on, the mean key row accumulates from
//           the same LDS tiles.
#include <math.h>
#include <stdlib.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <random>

#include "ikv_internal.hpp"
#include "res_setup.hpp"

namespace ikv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int MD = 128;          // head dimension of this path
constexpr int KROW = MD + 8;     // LDS row stride in bf16 (272 B): 16-lane column reads hit 64 distinct banks
constexpr float LOG2E = 1.4426950408889634f;

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// M' = M * log2(e) / sqrt(D) split into bf16 hi and lo. Per (unit, row), 256 bf16
// in fragment order [g 0..3][k-step 0..3][hi 8 | lo 8], where (k-step, g) holds
// channels (4 k-step + g) * 8 .. + 8: lane group g of an MFMA reads 128 contiguous bytes.
// Each unit's rows are padded to whole 16-row slices (pad16), the pad rows zero.
// Workgroup p takes padded rows [p*rows/P, (p+1)*rows/P) with P = MBAR_PARTS; thread (r, c)
// splits channel group c of rows r, r + 16, ... (32 bytes in, two 16-byte stores out),
// a batch of rows in flight at once (loads from row indices clamped into the range and
// masked afterwards, so that none waits inside a branch). With the residual head on it
// also sums the raw rows: the workgroup's column sums are partial p of mbar. For a
// session at or under its budget it only fills the scores with -inf (the gate).
constexpr int MS_BATCH = 9;

__global__ void __launch_bounds__(256) k_msplit(const ikv_session *__restrict__ sess, const float *__restrict__ M,
                                                float *__restrict__ ws, float *__restrict__ scores, int L, int Hkv,
                                                bool resid) {
  __shared__ float red[16][MD];
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  const int p = blockIdx.x;
  if (s.N <= s.C) {
    for (int j = p * 256 + int(threadIdx.x); j < s.N; j += MBAR_PARTS * 256) scores[s.slot_off + j] = -INFINITY;
    return;
  }
  const int units = L * Hkv;
  const int R = s.R, R16 = pad16(R);
  const int64_t rows = int64_t(units) * R16;
  const int64_t r0 = rows * p / MBAR_PARTS, r1 = rows * (p + 1) / MBAR_PARTS;
  const int rg = threadIdx.x >> 4, c = threadIdx.x & 15;
  const int g = c & 3, ks = c >> 2;
  const float scale = LOG2E / sqrtf(float(MD));
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  uint16_t *dst = reinterpret_cast<uint16_t *>(base) + (g * 4 + ks) * 16;
  const float *src = M + s.mem_off + c * 8;
  float cs[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) cs[e] = 0.f;
  for (int64_t r = r0 + rg; r < r1; r += 16 * MS_BATCH) {
    float4 va[MS_BATCH], vb[MS_BATCH];
#pragma unroll
    for (int k = 0; k < MS_BATCH; ++k) {
      const int64_t rr = min(r + 16 * k, r1 - 1);
      const int64_t u = rr / R16, row = min<int64_t>(rr - u * R16, R - 1);   // pad rows read the last row
      va[k] = *reinterpret_cast<const float4 *>(src + (u * R + row) * MD);
      vb[k] = *reinterpret_cast<const float4 *>(src + (u * R + row) * MD + 4);
    }
#pragma unroll
    for (int k = 0; k < MS_BATCH; ++k) {
      const int64_t rr = r + 16 * k;
      if (rr >= r1) continue;
      const bool real = rr - (rr / R16) * R16 < R;
      float v[8] = {va[k].x, va[k].y, va[k].z, va[k].w, vb[k].x, vb[k].y, vb[k].z, vb[k].w};
      if (!real)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        const float x0 = v[e] * scale, x1 = v[e + 1] * scale;
        const uint16_t h0 = float_to_bf16_bits(x0), h1 = float_to_bf16_bits(x1);
        const uint16_t l0 = float_to_bf16_bits(x0 - bf16_bits_to_float(h0));
        const uint16_t l1 = float_to_bf16_bits(x1 - bf16_bits_to_float(h1));
        hw[e / 2] = uint32_t(h0) | (uint32_t(h1) << 16);
        lw[e / 2] = uint32_t(l0) | (uint32_t(l1) << 16);
        cs[e] += v[e];
        cs[e + 1] += v[e + 1];
      }
      uint16_t *d = dst + rr * 256;
      *reinterpret_cast<uint4 *>(d) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
      *reinterpret_cast<uint4 *>(d + 8) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
    }
  }
  if (!resid) return;
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rg][c * 8 + e] = cs[e];
  __syncthreads();
  if (threadIdx.x < MD) {
    float tsum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) tsum += red[k][threadIdx.x];
    const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
    base[z.off_misc() + int64_t(p) * MD + threadIdx.x] = tsum;
  }
}

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// Sum over the 16 lanes of a row (lanes 16 q .. 16 q + 15), left in every lane of the row,
// by DPP lane moves instead of LDS permutes: quad_perm [1,0,3,2] and [2,3,0,1] add within
// each quad, row_half_mirror adds the other quad of the half row, row_mirror the other
// half. Each step adds a commutative pair, so every lane holds the same bits.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);                            // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);                            // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);                           // row_half_mirror
  v += dpp_mov<0x140>(v);                           // row_mirror
  return v;
}

constexpr int RING = 4;                          // LDS stages of key rows
constexpr int STAGE = MFMA_TILE * MD;            // bf16 per stage (32 KB)

// 16 bytes per lane from global memory straight into LDS at lds_base + 16 * lane.
// Issued from asm so that the compiler does not serialise LDS reads behind every
// outstanding load; the waits on these loads are placed by hand.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds_base), "v"(g)
               : "memory", "m0");
}
// The same with the non-temporal hint, for the key streams: a key row is read once
// per pass, and kept in L2 it would push out what the workgroups read again (the
// memory rows, which every workgroup of a head pair or unit reloads). Measured at
// Qwen3-8B 32k: first pass 443 -> 412 us, second pass 486 -> 435 us.
__device__ __forceinline__ void dma16_nt(const void *g, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt"
               :
               : "s"(lds_base), "v"(g)
               : "memory", "m0");
}

template <bool PASS_B, bool KBAR>
__global__ void __launch_bounds__(256) k_score_mfma(const uint16_t *__restrict__ kpool, int64_t num_slots, int L,
                                                    int Hkv, int dead, const ikv_session *__restrict__ sess,
                                                    const int32_t *__restrict__ slot_maps, float *__restrict__ ws,
                                                    float *__restrict__ scores, bool resid) {
  __shared__ __align__(1024) uint16_t kt[RING * STAGE];
  __shared__ int cand_s[MFMA_TILE];
  __shared__ float red[4][MFMA_TILE];

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int tile = blockIdx.x;
  const int j0 = tile * MFMA_TILE;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int R = s.R, R16 = pad16(R), nsl = R16 >> 4;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const uint16_t *msplit = reinterpret_cast<const uint16_t *>(base);
  float *part = base + z.off_part();
  const float *lse = base + z.off_lse();

  if (t < MFMA_TILE) {
    const int j = j0 + t;
    int c = 0;
    if (j < s.N) {
      const int slot = slot_maps[s.slot_off + j];
      c = slot != dead && !(j < s.pi || (j >= s.qs && j < s.qe));
    }
    cand_s[t] = c;
  }

  // DMA mapping: wave w, instruction k loads positions (8w + k)*4 + lane/16, 16-byte
  // slot lane%16 of the row, which holds chunk (lane%16) ^ (position%16).
  const uint32_t lds0 = uint32_t(reinterpret_cast<uintptr_t>(kt));
  const int64_t slot_stride = int64_t(Hkv) * MD;
  const uint16_t *src[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int tok = (8 * w + k) * 4 + (lane >> 4);
    const int j = j0 + tok;
    const int slot = j < s.N ? slot_maps[s.slot_off + j] : dead;     // past the end: any valid row
    const int chunk = (lane & 15) ^ (tok & 15);
    src[k] = kpool + int64_t(slot) * slot_stride + chunk * 8;
  }
  auto issue = [&](int u) {
    const int l = u / Hkv, h = u - l * Hkv;
    const int64_t off = int64_t(l) * num_slots * slot_stride + int64_t(h) * MD;
    const uint32_t st = lds0 + uint32_t((u % RING) * STAGE * 2);
#pragma unroll
    for (int k = 0; k < 8; ++k)
      dma16_nt(src[k] + off, __builtin_amdgcn_readfirstlane(st + uint32_t(((8 * w + k) * 4) * MD * 2)));
  };
  auto mload = [&](int u, bf16x8 (&mh)[4], bf16x8 (&ml)[4], int sl) {
    if (u >= units || sl >= nsl) return;
    const uint16_t *mp = msplit + (int64_t(u) * R16 + sl * 16 + (lane & 15)) * 256 + (lane >> 4) * 64;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      mh[ks] = *reinterpret_cast<const bf16x8 *>(mp + ks * 16);
      ml[ks] = *reinterpret_cast<const bf16x8 *>(mp + ks * 16 + 8);
    }
  };

  float racc[8][4];
  float kb[64];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int k = 0; k < 4; ++k) racc[i][k] = 0.f;
#pragma unroll
  for (int i = 0; i < 64; ++i) kb[i] = 0.f;

  auto compute = [&](int u, const uint16_t *kl, const bf16x8 (&mh0)[4], const bf16x8 (&ml0)[4]) {
    for (int sl = w; sl < nsl; sl += 4) {
      const int row = sl * 16 + (lane & 15);
      bf16x8 mh[4], ml[4];
      if (sl == w) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          mh[ks] = mh0[ks];
          ml[ks] = ml0[ks];
        }
      } else {
        mload(u, mh, ml, sl);
      }
      f32x4 acc[MFMA_TILE / 16];
#pragma unroll
      for (int blk = 0; blk < MFMA_TILE / 16; ++blk) {
        acc[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int tok = blk * 16 + (lane & 15);
        const uint16_t *kr = kl + tok * MD;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int chunk = 4 * ks + (lane >> 4);
          const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kr + ((chunk ^ (tok & 15)) * 8));
          acc[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, mh[ks], acc[blk], 0, 0, 0);
          acc[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, ml[ks], acc[blk], 0, 0, 0);
        }
      }
      // acc[blk][i]: position blk*16 + 4*(lane >> 4) + i, memory row `row`
      if (!PASS_B) {
        float m = -INFINITY;
#pragma unroll
        for (int blk = 0; blk < MFMA_TILE / 16; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (!cand_s[blk * 16 + 4 * (lane >> 4) + i]) acc[blk][i] = -INFINITY;
            m = fmaxf(m, acc[blk][i]);
          }
        const float mb = (m == -INFINITY) ? 0.f : m;
        float zs = 0.f;
#pragma unroll
        for (int blk = 0; blk < MFMA_TILE / 16; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) zs += ex2(acc[blk][i] - mb);
#pragma unroll
        for (int o = 16; o < 64; o <<= 1) {
          const float m2 = __shfl_xor(m, o, WAVE);
          const float z2 = __shfl_xor(zs, o, WAVE);
          const float mm = fmaxf(m, m2);
          const float a = (m == -INFINITY) ? 0.f : zs * ex2(m - mm);
          const float c = (m2 == -INFINITY) ? 0.f : z2 * ex2(m2 - mm);
          m = mm;
          zs = a + c;
        }
        if (lane < 16 && row < R) {                 // pad rows of the last slice are not stored
          float *p = part + ((int64_t(tile) * units + u) * R + row) * 2;
          p[0] = m;
          p[1] = zs;
        }
      } else {
        const int rowc = min(row, R - 1);
        const float mrow = lse[(int64_t(u) * R + rowc) * 2];
        const float iz = row < R ? lse[(int64_t(u) * R + rowc) * 2 + 1] : 0.f;   // pad rows add nothing
#pragma unroll
        for (int blk = 0; blk < MFMA_TILE / 16; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float p = ex2(acc[blk][i] - mrow) * iz;
            racc[blk][i] += cand_s[blk * 16 + 4 * (lane >> 4) + i] ? p : 0.f;
          }
      }
    }
    if (KBAR) {
      const int tok = 32 * w + (lane & 31);
      const uint16_t *kr = kl + tok * MD;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int chunk = (lane >> 5) * 8 + i;
        const uint4 v = *reinterpret_cast<const uint4 *>(kr + ((chunk ^ (tok & 15)) * 8));
        kb[8 * i + 0] += bf_lo(v.x);
        kb[8 * i + 1] += bf_hi(v.x);
        kb[8 * i + 2] += bf_lo(v.y);
        kb[8 * i + 3] += bf_hi(v.y);
        kb[8 * i + 4] += bf_lo(v.z);
        kb[8 * i + 5] += bf_hi(v.z);
        kb[8 * i + 6] += bf_lo(v.w);
        kb[8 * i + 7] += bf_hi(v.w);
      }
    }
  };

  // Unit u waits until its own 8 loads have landed: at most the loads of the later
  // units already issued (8 each) may still be in flight. Other vector-memory ops
  // issued in between only make the wait longer, never too short.
  auto wait_unit = [&](int u) {
    const int later = min(RING - 2, units - 1 - u);
    if (later >= 2) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
    else if (later == 1) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };

  bf16x8 mh0[4], ml0[4], mh1[4], ml1[4];
  for (int u = 0; u < RING - 1 && u < units; ++u) issue(u);
  mload(0, mh0, ml0, w);
  mload(1, mh1, ml1, w);
  for (int u = 0; u < units; u += 2) {
    wait_unit(u);
    __syncthreads();
    if (u + RING - 1 < units) issue(u + RING - 1);
    compute(u, kt + (u % RING) * STAGE, mh0, ml0);
    mload(u + 2, mh0, ml0, w);
    if (u + 1 >= units) break;
    wait_unit(u + 1);
    __syncthreads();
    if (u + RING < units) issue(u + RING);
    compute(u + 1, kt + ((u + 1) % RING) * STAGE, mh1, ml1);
    mload(u + 3, mh1, ml1, w);
  }
  __syncthreads();

  if (PASS_B) {
#pragma unroll
    for (int blk = 0; blk < MFMA_TILE / 16; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = racc[blk][i];
        v += __shfl_xor(v, 1, WAVE);
        v += __shfl_xor(v, 2, WAVE);
        v += __shfl_xor(v, 4, WAVE);
        v += __shfl_xor(v, 8, WAVE);
        if ((lane & 15) == 0) red[w][blk * 16 + 4 * (lane >> 4) + i] = v;
      }
    __syncthreads();
    if (t < MFMA_TILE) {
      const int j = j0 + t;
      if (j < s.N)
        scores[s.slot_off + j] = cand_s[t] ? (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]) : -INFINITY;
    }
  }
  if (KBAR) {
    const int tok = 32 * w + (lane & 31);
    const int j = j0 + tok;
    if (j < s.N) {
      const float inv = 1.0f / float(units);
      float *dst = base + z.off_kbar() + int64_t(j) * MD + (lane >> 5) * 64;
#pragma unroll
      for (int e = 0; e < 64; e += 4)
        *reinterpret_cast<float4 *>(dst + e) = make_float4(kb[e] * inv, kb[e + 1] * inv, kb[e + 2] * inv,
                                                           kb[e + 3] * inv);
    }
  }
}

// ------------------------------------------------------------------ first pass, position-major (R <= 64, odd Hkv)
// Keys and memory rows both stream by direct global->LDS loads: three 32 KB key
// stages and two 32 KB memory stages fill the 160 KB of LDS. With no compiler-issued
// vector loads left in the unit loop, the waits placed by hand are the only ones.
// Eight waves, two per SIMD: wave w takes the 16 memory rows of slice w & 3 against
// the 64 positions of half w >> 2, so one wave's LDS reads and exp2 run under the
// other's MFMAs. Each (64 positions, unit, row) leaves one (max, sum) in the log2
// domain. The unit-major pass below is used instead whenever Hkv is even.
constexpr int KSTAGES = 3;
constexpr int MSTAGE = 64 * 256;                 // bf16 per memory stage: 64 rows x 512 B

// s_waitcnt vmcnt(n) for a wave-uniform n in 0..12
__device__ __forceinline__ void vm_wait(int n) {
  switch (n) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(2)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(6)" ::: "memory"); break;
    case 8: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
    case 10: asm volatile("s_waitcnt vmcnt(10)" ::: "memory"); break;
    case 12: asm volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
  }
}

constexpr int RING_THREADS = 512;

// Read-only view for wave-uniform loads: the compiler issues them on the scalar unit.
typedef const __attribute__((address_space(4))) float cfloat;

__global__ void __launch_bounds__(RING_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_score_ring(const uint16_t *__restrict__ kpool, int64_t num_slots, int L, int Hkv, int dead,
             const ikv_session *__restrict__ sess, const int32_t *__restrict__ slot_maps, float *__restrict__ ws,
             bool resid) {
  __shared__ __align__(1024) uint16_t lds[KSTAGES * STAGE + 2 * MSTAGE];

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int tile = blockIdx.x;
  const int j0 = tile * MFMA_TILE;
  if (j0 >= s.N) return;
  const int units = L * Hkv;
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);   // wave-uniform: branches on it stay scalar
  const int rs = w & 3, half = w >> 2;             // memory-row slice, position half
  const int g = lane >> 4, r16 = lane & 15;
  const int R = s.R, R16 = pad16(R), nsl = R16 >> 4;
  const bool act = rs < nsl;
  const int row = rs * 16 + r16;
  const int p0 = half * 64;                        // first position of this wave's half
  const int ptile = tile * 2 + half;
  const bool pstore = act && lane < 16 && row < R && int64_t(ptile) * PART_TILE < s.N;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const uint16_t *msplit = reinterpret_cast<const uint16_t *>(base);
  float *part = base + z.off_part();
  const int32_t *S = slot_maps + s.slot_off;

  // candidate flags of this lane's 16 MFMA outputs: bit blk*4 + i <-> position p0 + blk*16 + 4g + i
  uint32_t cmask = 0;
#pragma unroll
  for (int blk = 0; blk < 4; ++blk)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = j0 + p0 + blk * 16 + 4 * g + i;
      if (j < s.N && S[j] != dead && !(j < s.pi || (j >= s.qs && j < s.qe))) cmask |= 1u << (blk * 4 + i);
    }

  // Key DMA: wave w, instruction k loads positions (4w + k)*4 + lane/16, 16-byte slot
  // lane%16 of the row, which holds chunk (lane%16) ^ (position%16).
  const uint32_t lds0 = uint32_t(reinterpret_cast<uintptr_t>(lds));
  const uint32_t mlds0 = lds0 + uint32_t(KSTAGES * STAGE * 2);
  const int64_t slot_stride = int64_t(Hkv) * MD;
  const uint16_t *src[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int tok = (4 * w + k) * 4 + (lane >> 4);
    const int j = j0 + tok;
    const int slot = j < s.N ? S[j] : dead;        // past the end: any valid row
    src[k] = kpool + int64_t(slot) * slot_stride + ((lane & 15) ^ (tok & 15)) * 8;
  }
  // every compiler-issued load of the set-up is complete before the first DMA
  asm volatile("" ::"v"(cmask), "v"(src[0]), "v"(src[1]), "v"(src[2]), "v"(src[3]));
  auto issue_k_piece = [&](int u, int k) {
    const int l = u / Hkv, h = u - l * Hkv;
    const int64_t off = int64_t(l) * num_slots * slot_stride + int64_t(h) * MD;
    const uint32_t st = lds0 + uint32_t((u % KSTAGES) * STAGE * 2);
    dma16_nt(src[k] + off, __builtin_amdgcn_readfirstlane(st + uint32_t(((4 * w + k) * 4) * MD * 2)));
  };
  auto issue_k = [&](int u) {
#pragma unroll
    for (int k = 0; k < 4; ++k) issue_k_piece(u, k);
  };
  // memory rows of unit u: R16 rows of 512 B (the pad rows zero), 32 chunks of 16 B per
  // row, chunk slot s of row r holds chunk s ^ (r & 15); wave w issues R16/16 of the
  // R16/2 1-KB pieces
  const int nm = R16 >> 4;
  auto issue_m_piece = [&](int u, int k) {
    const uint16_t *m0 = msplit + int64_t(u) * R16 * 256;
    const uint32_t st = mlds0 + uint32_t((u & 1) * MSTAGE * 2);
    const int piece = w * nm + k;
    const int r = piece * 2 + (lane >> 5);
    const int sl = lane & 31;
    dma16(m0 + r * 256 + ((sl ^ (r & 15)) * 8), __builtin_amdgcn_readfirstlane(st + uint32_t(piece * 1024)));
  };
  // The loads of the next stages during unit u, spread over its eight MFMA chunks: the
  // memory-row pieces of unit u + 1 in chunks 0-1, the key pieces of unit u + 2 in
  // chunks 2-5. The order (memory rows first) keeps the count the top of each unit
  // waits for.
  auto dma_chunk = [&](int u, int c) {
    if (c < 2) {
#pragma unroll
      for (int k = 2 * c; k < 2 * c + 2; ++k)
        if (k < nm && u + 1 < units) issue_m_piece(u + 1, k);
    } else if (c < 6) {
      if (u + 2 < units) issue_k_piece(u + 2, c - 2);
    }
  };

  float pm = 0.f, pz = 0.f;                        // the previous unit's (max, sum)
  // The logits of a unit are finished (masked max and sum) during the next unit, on
  // the VALU under that unit's MFMAs: the two pipes overlap, and the epilogue reads
  // only registers, so it may cross the barrier.
  f32x4 accp[4];
#pragma unroll
  for (int blk = 0; blk < 4; ++blk) accp[blk] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  // Epilogue of one unit in eight steps, so that each step can run under four MFMAs
  // of the next unit: masked max (step 0), exp2 sums (steps 1-4), the merge across the
  // four lane groups of a row (steps 5-6).
  float em = -INFINITY, emb = 0.f, ez = 0.f;
  auto epilogue_step = [&](f32x4 (&a)[4], int c) {
    if (c == 0) {
      em = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (!((cmask >> (blk * 4 + i)) & 1u)) a[blk][i] = -INFINITY;
          em = fmaxf(em, a[blk][i]);
        }
      emb = (em == -INFINITY) ? 0.f : em;
      ez = 0.f;
    } else if (c <= 4) {
#pragma unroll
      for (int i = 0; i < 4; ++i) ez += ex2(a[c - 1][i] - emb);
    } else if (c <= 6) {
      const int o = c == 5 ? 16 : 32;
      const float m2 = __shfl_xor(em, o, WAVE);
      const float z2 = __shfl_xor(ez, o, WAVE);
      const float mm = fmaxf(em, m2);
      const float x = (em == -INFINITY) ? 0.f : ez * ex2(em - mm);
      const float y = (m2 == -INFINITY) ? 0.f : z2 * ex2(m2 - mm);
      em = mm;
      ez = x + y;
      if (c == 6) {
        pm = em;
        pz = ez;
      }
    }
  };
  auto epilogue = [&](f32x4 (&a)[4]) {
#pragma unroll
    for (int c = 0; c < 8; ++c) epilogue_step(a, c);
  };

  auto compute = [&](int u) {
    const uint16_t *kl = lds + (u % KSTAGES) * STAGE;
    if (act) {
      const uint16_t *mr = lds + KSTAGES * STAGE + (u & 1) * MSTAGE + row * 256;
      // fragments of k-step ks: memory row hi/lo and the four key blocks; k-step 0 now,
      // each later one two chunks before its MFMAs, so that the eight waves' LDS reads
      // spread over the unit instead of all landing at its start
      bf16x8 mh[4], ml[4], ka[4][4];
      auto read_ks = [&](int ks) {
        mh[ks] = *reinterpret_cast<const bf16x8 *>(mr + (((g * 8 + ks * 2) ^ r16) * 8));
        ml[ks] = *reinterpret_cast<const bf16x8 *>(mr + (((g * 8 + ks * 2 + 1) ^ r16) * 8));
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
          ka[blk][ks] = *reinterpret_cast<const bf16x8 *>(kl + (p0 + blk * 16 + r16) * MD + (((4 * ks + g) ^ r16) * 8));
      };
      dma_chunk(u, 0);
      read_ks(0);
      f32x4 acc[4];
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) acc[blk] = f32x4{0.f, 0.f, 0.f, 0.f};
      // chunk c: the four MFMAs of k-step c/2 (hi, then lo), then epilogue step c of
      // the previous unit (a no-op before the first); the fences keep the interleave
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int ks = c >> 1;
        if (c > 0) dma_chunk(u, c);
        if ((c & 1) == 0 && ks + 1 < 4) read_ks(ks + 1);
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
          acc[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[blk][ks], (c & 1) ? ml[ks] : mh[ks], acc[blk], 0, 0, 0);
        epilogue_step(accp, c);
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) accp[blk] = acc[blk];
    } else {
#pragma unroll
      for (int c = 0; c < 6; ++c) dma_chunk(u, c);
    }
  };
  auto store_part = [&](int u) {
    if (pstore)
      *reinterpret_cast<float2 *>(part + ((int64_t(ptile) * units + u) * R + row) * 2) = make_float2(pm, pz);
  };

  // Issue order per wave: K(0), M(0), K(1), then per unit u: the store of unit u-2,
  // M(u+1), K(u+2), the last two spread over the unit's MFMA chunks. At the top of
  // unit u only K(u+1) (4 loads) may still be younger than M(u) and K(u).
  issue_k(0);
  for (int k = 0; k < nm; ++k) issue_m_piece(0, k);
  if (units > 1) issue_k(1);
  for (int u = 0; u < units; ++u) {
    if (u + 1 < units) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (u >= 2) store_part(u - 2);                 // finished during unit u - 1
    compute(u);
  }
  if (units >= 2) store_part(units - 2);
  if (act) epilogue(accp);                         // the last unit
  store_part(units - 1);
}

// ------------------------------------------------------------------ second pass, warp-specialised (R <= 64)
// The second pass as producer and consumer waves. A wave that issues a load into LDS can
// stall until the CU's address unit takes it, and the ring's 64 KB per unit keep that unit
// busy most of the time; when the waves that issue the loads are also the ones running the
// MFMAs, those stalls leave the matrix cores idle. Here waves 4-7 (producers) issue every
// load of the ring and sum the mean key row on the VALU; waves 0-3 (consumers, one per
// SIMD) only read LDS, run the logit MFMAs and fold exp2 of the logits into the rule score.
// Consumer c takes memory rows 32 (c & 1) .. + 31 against positions 64 (c >> 1) .. + 63,
// which reads 128 KB of LDS per unit instead of the 192 KB of sixteen-row waves.
constexpr int WS_THREADS = 512;

// RH row halves per unit: 1 for sessions of up to 64 memory rows; 2 for up to 128,
// where every unit's rows stream as two halves of 64 through the same two-stage ring
// (half h in stage h) against the one key stage of the unit. A batch holding both
// kinds runs one launch of each; `big` as in k_score_stats.
//
// STASH (every session R <= 16, one row slice): the one-key-pass form. The producers run
// unchanged (keys, the 16 split rows, the mean key row); consumer c takes entries
// 32 c .. + 31 against the slice and, per unit, stores the raw logits (log2 domain) to the
// stash and merges the tile's (max, sum of exp2) per row across the four consumers,
// written as the list tile's partial (chunk-major, c per + k, whatever the grid order);
// k_lse_mfma and k_score_stash finish the score.
template <bool KBAR, int RH, bool STASH = false>
__global__ void __launch_bounds__(WS_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_score_ws(const uint16_t *__restrict__ kpool, int64_t num_slots, int L, int Hkv, int dead,
           const ikv_session *__restrict__ sess, const int32_t *__restrict__ slot_maps, float *__restrict__ ws,
           float *__restrict__ scores, bool resid, int big, int CH) {
  __shared__ __align__(1024) uint16_t lds[KSTAGES * STAGE + 2 * MSTAGE];

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  if ((big == 1 && s.R > 64) || (big == 2 && s.R <= 64)) return;   // the other launch's session
  // list tile k of chunk c covers entries [c CH + 128 k, + 128) of the candidate list. The
  // grid runs tile-index-major (block x = k * chunks + c): chunk-major, tile k of every
  // chunk would land on XCD k, and a session whose chunks hold few candidates would pile
  // its work onto the first XCDs while the empty tiles of the others finish at once.
  const int per = CH / MFMA_TILE, nch = int(gridDim.x) / per;
  const int lc = int(blockIdx.x) % nch, lk = int(blockIdx.x) / nch;
  if (int64_t(lc) * CH >= s.N) return;
  const int units = L * Hkv;
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int g = lane >> 4, r16 = lane & 15;
  const int R = s.R, R16 = pad16(R);
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const int32_t *S = slot_maps + s.slot_off;
  const uint32_t lds0 = uint32_t(reinterpret_cast<uintptr_t>(lds));
  const int32_t *lst = reinterpret_cast<const int32_t *>(base + z.off_clist()) + lc * CH + lk * MFMA_TILE;
  const int cnt = reinterpret_cast<const int32_t *>(base + z.off_ccount(s.N))[lc];
  const int ne = min(MFMA_TILE, cnt - lk * MFMA_TILE);
  if (ne <= 0) {
    if constexpr (STASH) {                           // an empty list tile still leaves its partials
      float2 *pt = reinterpret_cast<float2 *>(base + z.off_part()) + (int64_t(lc) * per + lk) * units * R;
      for (int i = t; i < units * R; i += WS_THREADS) pt[i] = make_float2(-INFINITY, 0.f);
    }
    return;
  }
  // a chunk whose every position is a candidate is its own list: entry e is position e0 + e
  const bool ident = cnt == min(CH, s.N - lc * CH);
  const int e0 = lc * CH + lk * MFMA_TILE;
  auto pos_of = [&](int e) __attribute__((always_inline)) { return ident ? e0 + e : lst[e]; };

  if (w >= 4) {
    // ---------------- producers: the ring's loads, and the mean key row
    const int pw = w - 4;
    const int64_t slot_stride = int64_t(Hkv) * MD;
    // key instruction k of producer pw loads positions (8 pw + k) * 4 + lane / 16, 16-byte
    // slot lane % 16 of the row, which holds chunk (lane % 16) ^ (position % 16)
    const uint16_t *src[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int tok = (8 * pw + k) * 4 + (lane >> 4);
      const int slot = tok < ne ? S[pos_of(tok)] : dead;   // past the list: any valid row
      src[k] = kpool + int64_t(slot) * slot_stride + ((lane & 15) ^ (tok & 15)) * 8;
    }
    asm volatile("" ::"v"(src[0]), "v"(src[7]));   // the slot loads are complete before the first DMA
    auto issue_k_piece = [&](int u, int k) __attribute__((always_inline)) {
      const int l = u / Hkv, h = u - l * Hkv;
      const int64_t off = int64_t(l) * num_slots * slot_stride + int64_t(h) * MD;
      const uint32_t st = lds0 + uint32_t((u % KSTAGES) * STAGE * 2);
      dma16_nt(src[k] + off, __builtin_amdgcn_readfirstlane(st + uint32_t(((8 * pw + k) * 4) * MD * 2)));
    };
    auto issue_k = [&](int u) __attribute__((always_inline)) {
#pragma unroll
      for (int k = 0; k < 8; ++k) issue_k_piece(u, k);
    };
    // memory rows of unit u (half hf): up to 64 rows of 512 B (R16 per unit, the pad rows
    // zero), chunk slot c of row r holds chunk c ^ (r & 15); producer pw issues a quarter
    // of the half's 1-KB pieces (two rows each), npc(hf) of them
    const uint16_t *msplit = reinterpret_cast<const uint16_t *>(base);
    const uint32_t mlds0 = lds0 + uint32_t(KSTAGES * STAGE * 2);
    auto npc_of = [&](int hf) __attribute__((always_inline)) { return min(64, max(0, R16 - 64 * hf)) >> 3; };
    auto issue_m_piece = [&](int u, int hf, int k) __attribute__((always_inline)) {
      const int npc = npc_of(hf);
      const uint16_t *m0 = msplit + (int64_t(u) * R16 + 64 * hf) * 256;
      const uint32_t st = mlds0 + uint32_t((RH == 1 ? (u & 1) : hf) * MSTAGE * 2);
      const int piece = pw * npc + k;
      const int r = piece * 2 + (lane >> 5);
      const int sl = lane & 31;
      dma16(m0 + r * 256 + ((sl ^ (r & 15)) * 8), __builtin_amdgcn_readfirstlane(st + uint32_t(piece * 1024)));
    };
    auto issue_m = [&](int u, int hf) __attribute__((always_inline)) {
      for (int k = 0; k < npc_of(hf); ++k) issue_m_piece(u, hf, k);
    };
    const int npc = npc_of(0);
    // mean key row: lane (position 32 pw + lane % 32, channels 64 (lane / 32) .. + 63)
    const int pp = 32 * pw + (lane & 31), hc = lane >> 5;
    float kb[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) kb[i] = 0.f;

    // Issue order: K(0), M(0), K(1), then per unit u: M(u+1), K(u+2). At the top of unit u
    // only K(u+1) (8 loads) may still be younger than M(u) and K(u). Within a unit the
    // loads alternate with the mean-key-row steps (memory-row pieces in steps 0-3, two
    // each, key pieces in steps 4-7), so that the VALU work fills the time a wave waits
    // for the address unit to take its next load.
    auto kbar_step = [&](const uint16_t *kr, int c) __attribute__((always_inline)) {
      const uint4 v = *reinterpret_cast<const uint4 *>(kr + (((8 * hc + c) ^ (pp & 15)) * 8));
      const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {                  // bf16 -> float is exact: the high half of the word
        kb[8 * c + 2 * e] += __uint_as_float(q[e] << 16);
        kb[8 * c + 2 * e + 1] += __uint_as_float(q[e] & 0xffff0000u);
      }
    };
    issue_k(0);
    issue_m(0, 0);
    if (units > 1) issue_k(1);
    if constexpr (RH == 1) {
      for (int u = 0; u < units; ++u) {
        if (u + 1 < units) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        const uint16_t *kr = lds + (u % KSTAGES) * STAGE + pp * MD;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          if (c < 4) {
#pragma unroll
            for (int k = 2 * c; k < 2 * c + 2; ++k)
              if (k < npc && u + 1 < units) issue_m_piece(u + 1, 0, k);
          } else if (u + 2 < units) {
            issue_k_piece(u + 2, 2 * (c - 4));
            issue_k_piece(u + 2, 2 * (c - 4) + 1);
          }
          if (KBAR) kbar_step(kr, c);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    } else {
      // Per half hf of unit u: the next half's rows (M(u, 1), then M(u + 1, 0)) in
      // steps 0-1, then key pieces 4 hf .. 4 hf + 3 of K(u + 2) in steps 2-3; the mean
      // key row takes channel chunks 4 hf .. 4 hf + 3. At the top of a half only the
      // key pieces issued after its rows may be outstanding: K(1) (8) at the first,
      // four after that, none once the keys run out.
      for (int u = 0; u < units; ++u)
        for (int hf = 0; hf < 2; ++hf) {
          const int after = hf == 0 ? (u == 0 ? (units > 1 ? 8 : 0) : (u + 1 < units ? 4 : 0))
                                    : (u + 2 < units ? 4 : 0);
          vm_wait(after);
          __syncthreads();
          const uint16_t *kr = lds + (u % KSTAGES) * STAGE + pp * MD;
          const int nu = hf == 0 ? u : u + 1, nh = hf ^ 1, nn = npc_of(nh);
#pragma unroll
          for (int c4 = 0; c4 < 4; ++c4) {
            if (c4 < 2) {
#pragma unroll
              for (int k = 4 * c4; k < 4 * c4 + 4; ++k)
                if (k < nn && nu < units) issue_m_piece(nu, nh, k);
            } else if (u + 2 < units) {
              issue_k_piece(u + 2, 4 * hf + 2 * (c4 - 2));
              issue_k_piece(u + 2, 4 * hf + 2 * (c4 - 2) + 1);
            }
            if (KBAR) kbar_step(kr, 4 * hf + c4);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
    }
    __syncthreads();                                 // the ring is free (matches the consumers)
    // The mean key rows go out through LDS, so that each store writes two whole
    // 512-byte rows: stored straight from the lanes, every line would leave L2 in
    // 16-byte pieces. Rows of 132 floats keep the lanes' writes on distinct banks;
    // the region starts past the consumers' reduction buffer.
    float *kt = reinterpret_cast<float *>(lds) + 2 * MFMA_TILE;
    constexpr int KT_ROW = MD + 4;
    if (KBAR) {
      const float inv = 1.0f / float(units);
#pragma unroll
      for (int q = 0; q < 16; ++q)
        *reinterpret_cast<float4 *>(kt + pp * KT_ROW + 64 * hc + 4 * q) =
            make_float4(kb[4 * q] * inv, kb[4 * q + 1] * inv, kb[4 * q + 2] * inv, kb[4 * q + 3] * inv);
    }
    __syncthreads();
    if (KBAR) {
      // producer pw stores positions 32 pw .. + 31: two rows (32 lanes x 16 B each) per instruction
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int pr = 32 * pw + 2 * q + (lane >> 5);
        const float4 v = *reinterpret_cast<const float4 *>(kt + pr * KT_ROW + 4 * (lane & 31));
        if (pr < ne) reinterpret_cast<float4 *>(base + z.off_kbar() + int64_t(pos_of(pr)) * MD)[lane & 31] = v;
      }
    }
    return;
  }

  if constexpr (STASH) {
    // ---------------- consumers, one-key-pass form: logits to the stash, per-tile row statistics
    const int q0 = 32 * w;                           // this consumer's 32 entries
    const int64_t NS = stash_stride(s.N);
    float *stash = base + z.off_stash() + int64_t(lc) * CH + int64_t(lk) * MFMA_TILE + q0 + 4 * g;
    float2 *pt = reinterpret_cast<float2 *>(base + z.off_part()) + (int64_t(lc) * per + lk) * units * R;
    // per-consumer (max, sum) of unit u's rows: [u & 1][consumer][row], in the first
    // memory stage's unused space past its 16 rows
    float2 *sb = reinterpret_cast<float2 *>(lds + KSTAGES * STAGE + 16 * 256);
    // consumer 0 merges unit u's four partials of each row < R into the tile's partial
    auto merge = [&](int u) __attribute__((always_inline)) {
      if (w == 0 && lane < R) {
        const float2 *q = sb + (u & 1) * 64 + lane;
        float m = -INFINITY;
#pragma unroll
        for (int c = 0; c < 4; ++c) m = fmaxf(m, q[16 * c].x);
        float zs = 0.f;
        if (m != -INFINITY)
#pragma unroll
          for (int c = 0; c < 4; ++c)
            if (q[16 * c].x != -INFINITY) zs += q[16 * c].y * ex2(q[16 * c].x - m);
        pt[int64_t(u) * R + lane] = make_float2(m, zs);
      }
    };
    for (int u = 0; u < units; ++u) {
      __syncthreads();                               // stage u in LDS; unit u - 1's partials in sb
      if (u > 0) merge(u - 1);
      const uint16_t *kl = lds + (u % KSTAGES) * STAGE;
      const uint16_t *mr = lds + KSTAGES * STAGE + (u & 1) * MSTAGE + r16 * 256;
      bf16x8 mh[4], ml[4], ka[2][4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        mh[ks] = *reinterpret_cast<const bf16x8 *>(mr + (((g * 8 + ks * 2) ^ r16) * 8));
        ml[ks] = *reinterpret_cast<const bf16x8 *>(mr + (((g * 8 + ks * 2 + 1) ^ r16) * 8));
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
          ka[blk][ks] = *reinterpret_cast<const bf16x8 *>(kl + (q0 + blk * 16 + r16) * MD + (((4 * ks + g) ^ r16) * 8));
      }
      // lane (g, r16) of block blk: row r16 at entries q0 + 16 blk + 4 g + i
      f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
          acc[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[blk][ks], mh[ks], acc[blk], 0, 0, 0);
          acc[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[blk][ks], ml[ks], acc[blk], 0, 0, 0);
        }
      if (r16 < R) {
        float *o = stash + (int64_t(u) * R + r16) * NS;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)         // read once, by k_score_stash: non-temporal
          __builtin_nontemporal_store(acc[blk], reinterpret_cast<f32x4 *>(o + 16 * blk));
      }
      // the row's max and sum over this consumer's entries below ne (the four lane groups
      // of a row combined by shuffles: a merge of per-lane partials by consumer 0 made it
      // the straggler at every unit's barrier, 0.49 against 0.37 ms per multi-turn call)
      float m = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (q0 + 16 * blk + 4 * g + i >= ne) acc[blk][i] = -INFINITY;
          m = fmaxf(m, acc[blk][i]);
        }
      m = fmaxf(m, __shfl_xor(m, 16, WAVE));
      m = fmaxf(m, __shfl_xor(m, 32, WAVE));
      float zs = 0.f;
      if (m != -INFINITY)
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
          for (int i = 0; i < 4; ++i) zs += ex2(acc[blk][i] - m);
      zs += __shfl_xor(zs, 16, WAVE);
      zs += __shfl_xor(zs, 32, WAVE);
      if (g == 0) sb[(u & 1) * 64 + 16 * w + r16] = make_float2(m, zs);
    }
    __syncthreads();                                 // matches the producers' "ring is free"
    merge(units - 1);
    __syncthreads();                                 // matches the producers' mean-key-row barrier
    return;
  }

  // ---------------- consumers: logits on the matrix cores, exp2 folded into the rule score
  const int rh = w & 1, p0 = (w >> 1) * 64;         // memory-row half, first position of the half
  const int nsl = R16 >> 4;
  const float *nl2 = base + z.off_nl2();
  float racc[4][4];
#pragma unroll
  for (int blk = 0; blk < 4; ++blk)
#pragma unroll
    for (int i = 0; i < 4; ++i) racc[blk][i] = 0.f;
  f32x4 accp[2][4];
#pragma unroll
  for (int sl = 0; sl < 2; ++sl)
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) accp[sl][blk] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
  // step c (0-7) of the previous unit's epilogue: exp2 of four of its 32 logits per lane
  auto epilogue_step = [&](int c) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int e = 4 * c + k, sl = e >> 4, blk = (e >> 2) & 3, i = e & 3;
      racc[blk][i] += ex2(accp[sl][blk][i]);
    }
  };
  // Seeds -(max + log2 Z) of the lane's two rows, loaded two (virtual) units ahead at
  // the end of a unit's MFMAs: issued right after the barrier, a load would queue behind
  // the producers' ring loads at the address unit. Rows past R take -inf against zero
  // fragments, so exp2 of their logits is 0. Virtual unit v is half v % RH of unit v / RH.
  auto rowv = [&](int v, int k) __attribute__((always_inline)) { return 64 * (v % RH) + 32 * rh + 16 * k + r16; };
  auto seed_ld = [&](int v, int k) __attribute__((always_inline)) { return nl2[int64_t(v / RH) * R + min(rowv(v, k), R - 1)]; };
  // one virtual unit: seeds s0, s1 as loaded (rows past R take -inf here)
  auto unit_step = [&](int v, float s0, float s1) __attribute__((always_inline)) {
    const int u = v / RH, hf = v % RH;
    const float seed0 = rowv(v, 0) < R ? s0 : -INFINITY, seed1 = rowv(v, 1) < R ? s1 : -INFINITY;
    const bool act0 = 4 * hf + 2 * rh < nsl, act1 = 4 * hf + 2 * rh + 1 < nsl;   // slices within R
    __syncthreads();
    const uint16_t *kl = lds + (u % KSTAGES) * STAGE;
    const uint16_t *mb = lds + KSTAGES * STAGE + (RH == 1 ? (u & 1) : hf) * MSTAGE;
    const uint16_t *mr0 = mb + (32 * rh + r16) * 256, *mr1 = mr0 + 16 * 256;
    // fragments of k-step ks: memory rows (hi, lo) of both slices, the four key blocks
    bf16x8 mh[2][4], ml[2][4], ka[4][4];
    auto read_ks = [&](int ks) __attribute__((always_inline)) {
      const int ch = ((g * 8 + ks * 2) ^ r16) * 8, cl = ((g * 8 + ks * 2 + 1) ^ r16) * 8;
      mh[0][ks] = *reinterpret_cast<const bf16x8 *>(mr0 + ch);
      ml[0][ks] = *reinterpret_cast<const bf16x8 *>(mr0 + cl);
      mh[1][ks] = *reinterpret_cast<const bf16x8 *>(mr1 + ch);
      ml[1][ks] = *reinterpret_cast<const bf16x8 *>(mr1 + cl);
      if (!act0) mh[0][ks] = ml[0][ks] = bf16x8{};
      if (!act1) mh[1][ks] = ml[1][ks] = bf16x8{};
#pragma unroll
      for (int blk = 0; blk < 4; ++blk)
        ka[blk][ks] = *reinterpret_cast<const bf16x8 *>(kl + (p0 + blk * 16 + r16) * MD + (((4 * ks + g) ^ r16) * 8));
    };
    read_ks(0);
    f32x4 acc[2][4];
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      acc[0][blk] = f32x4{seed0, seed0, seed0, seed0};
      acc[1][blk] = f32x4{seed1, seed1, seed1, seed1};
    }
    // chunk c: the eight MFMAs of k-step c/2 (hi, then lo) for both slices, then step c of
    // the previous unit's epilogue; the fences keep the interleave
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int ks = c >> 1;
      if ((c & 1) == 0 && ks + 1 < 4) read_ks(ks + 1);
#pragma unroll
      for (int sl = 0; sl < 2; ++sl)
#pragma unroll
        for (int blk = 0; blk < 4; ++blk)
          acc[sl][blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[blk][ks], (c & 1) ? ml[sl][ks] : mh[sl][ks],
                                                                 acc[sl][blk], 0, 0, 0);
      epilogue_step(c);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int sl = 0; sl < 2; ++sl)
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) accp[sl][blk] = acc[sl][blk];
  };
  // Even and odd virtual units keep their own seed registers (unrolled by two), so
  // that no register that a load is still filling has to be copied.
  const int V = units * RH;
  float a0 = seed_ld(0, 0), a1 = seed_ld(0, 1), b0 = 0.f, b1 = 0.f;
  if (V > 1) {
    b0 = seed_ld(1, 0);
    b1 = seed_ld(1, 1);
  }
  for (int v = 0; v < V; v += 2) {
    unit_step(v, a0, a1);
    if (v + 2 < V) {
      a0 = seed_ld(v + 2, 0);
      a1 = seed_ld(v + 2, 1);
    }
    if (v + 1 < V) {
      unit_step(v + 1, b0, b1);
      if (v + 3 < V) {
        b0 = seed_ld(v + 3, 0);
        b1 = seed_ld(v + 3, 1);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) epilogue_step(c);      // the last unit
  __syncthreads();                                   // the ring is free: reuse it for the reduction
  float *red = reinterpret_cast<float *>(lds);       // [2][MFMA_TILE]
#pragma unroll
  for (int blk = 0; blk < 4; ++blk)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = racc[blk][i];                        // position p0 + 16 blk + 4 g + i, row r16 of both slices
      v += __shfl_xor(v, 1, WAVE);
      v += __shfl_xor(v, 2, WAVE);
      v += __shfl_xor(v, 4, WAVE);
      v += __shfl_xor(v, 8, WAVE);
      if (r16 == 0) red[rh * MFMA_TILE + p0 + blk * 16 + 4 * g + i] = v;
    }
  __syncthreads();
  if (t < ne) scores[s.slot_off + pos_of(t)] = red[t] + red[MFMA_TILE + t];   // every list entry is a candidate
}

// ------------------------------------------------------------------ one key pass at R <= 64
// k_score_fused: the rule score of Eq. 3 with one read of the keys, for a session whose
// list tiles all fit on the device at once (one workgroup per tile, cooperative launch).
// Eq. 3 needs each memory row's normaliser over every candidate before any score, and a
// tile's workgroup sees only its own 128 positions. So for every unit the workgroups
// exchange per-row partials while they go on: a tile computes unit v's logits, keeps
// e = exp2(x - m) of its 64 positions per row (m its own row maximum) and publishes
// (m, sum e); FU_LAG units later the row normaliser c = max + log2 Z of that unit is in,
// and the tile adds exp2(m - c) * e over the rows to each position's score.
//
// Producers (waves 4-7) are the second pass's: the key and memory-row rings and the mean
// key row. Producer 3 also combines the rows it owns: row r of unit x belongs to
// workgroup (x * R16 + r) mod G, one row every G / R16 units. At the top of a unit it
// checks the partials its loads of the previous top returned, stores the row's stamped
// normaliser when every partial is in and reissues the loads when not; it waits only
// when the row is due (at the top of unit x + FU_LAG, the last top before a tile
// finishes unit x).
// Consumers (waves 0-3): wave c takes memory rows 32 (c & 1) .. + 31 against entries
// 64 (c >> 1) .. + 63, as two 32 x 32 blocks of v_mfma_f32_32x32x16_bf16 (keys as A,
// split memory rows as B, hi then lo): lane l holds row 32 (c & 1) + l % 32 and 32
// entries. Unit v's step: finish unit v - 1 - FU_LAG (its normaliser loaded at the
// previous step; the weighted rows reduce-scatter over the 32 lanes of a half, so each
// lane keeps one entry's running score), then unit v's MFMAs with unit v - 1's row
// statistics and exp2 folded in between. Five 32-register slots rotate over the units.
//
// Exchange words (device scope, 64 bits, never cached non-coherently): partial
// (unit u, row r, half q) = {m | lo(S_u)}, {sum | hi(S_u)} and normaliser (u, r) =
// {c | lo(S_u)}, {c | hi(S_u)}, S_u = stamp + u, a 64-bit stamp the host draws per call
// (a random per-process tag above a call counter), so leftovers of other calls and of
// other data never pass. Every wait is bounded (`spins` polls); one that runs out sets
// the host fault word, which the library's next call reports as IKV_EHIP.
//
// The form is switched off (fused_tiles: a wrong normaliser on some calls, cause not
// found). Where it ran, at the Qwen3-8B 32k shape a normaliser landed 7-12 us after its
// unit's last partial, while FU_LAG units of work take about 6 us, so the tiles waited at
// almost every unit and the call was slower than the two key passes.
constexpr bool FU_ENABLED = false;               // see fused_tiles
constexpr int FU_LAG = 4;
constexpr int FU_SLOTS = FU_LAG + 1;
constexpr int FU_MIN_TILES = 64;                 // >= 64 rows per unit: one owned row per unit at most
constexpr int FU_MAX_TILES = 256;                // partials per owner lane: at most 8

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void fu_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ u32x4 ld_coherent16(const void *p) {
  u32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ void st_word(uint64_t *p, float v, uint32_t tag) {
  __hip_atomic_store(p, (uint64_t(__float_as_uint(v)) << 32) | tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_word(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <bool KBAR>
__global__ void __launch_bounds__(WS_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_score_fused(const uint16_t *__restrict__ kpool, int64_t num_slots, int L, int Hkv, int dead,
              const ikv_session *__restrict__ sess, const int32_t *__restrict__ slot_maps, float *__restrict__ ws,
              float *__restrict__ scores, bool resid, int CH, uint64_t *__restrict__ xch, uint64_t stamp,
              uint32_t spins, uint32_t *__restrict__ host_fault) {
  __shared__ __align__(1024) uint16_t lds[KSTAGES * STAGE + 2 * MSTAGE];

  const ikv_session s = sess[0];
  if (s.N <= s.C) return;                          // every workgroup alike: no event
  const int G = int(gridDim.x), wgi = int(blockIdx.x);
  const int per = CH / MFMA_TILE, nch = G / per;
  const int lc = wgi % nch, lk = wgi / nch;
  const int units = L * Hkv;
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int R = s.R, R16 = pad16(R);
  const int P = 2 * G;                             // partials per (unit, row)
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, 0, L, units, MD, resid, true);
  const int32_t *S = slot_maps + s.slot_off;
  const uint32_t lds0 = uint32_t(reinterpret_cast<uintptr_t>(lds));
  const int32_t *lst = reinterpret_cast<const int32_t *>(base + z.off_clist()) + lc * CH + lk * MFMA_TILE;
  const int cnt = reinterpret_cast<const int32_t *>(base + z.off_ccount(s.N))[lc];
  const int ne = max(0, min(MFMA_TILE, cnt - lk * MFMA_TILE));   // an empty tile still takes part
  const bool ident = cnt == min(CH, s.N - lc * CH);
  const int e0 = lc * CH + lk * MFMA_TILE;
  auto pos_of = [&](int e) __attribute__((always_inline)) { return ident ? e0 + e : lst[e]; };
  uint64_t *xpart = xch;
  uint64_t *xnrm = xch + int64_t(units) * R16 * P * 2;
  bool timed_out = false;

  if (w >= 4) {
    // ---------------- producers: the rings and the mean key row (as the second pass)
    const int pw = w - 4;
    const int64_t slot_stride = int64_t(Hkv) * MD;
    const uint16_t *src[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int tok = (8 * pw + k) * 4 + (lane >> 4);
      const int slot = tok < ne ? S[pos_of(tok)] : dead;   // past the list: any valid row
      src[k] = kpool + int64_t(slot) * slot_stride + ((lane & 15) ^ (tok & 15)) * 8;
    }
    asm volatile("" ::"v"(src[0]), "v"(src[7]));
    auto issue_k_piece = [&](int u, int k) __attribute__((always_inline)) {
      const int l = u / Hkv, h = u - l * Hkv;
      const int64_t off = int64_t(l) * num_slots * slot_stride + int64_t(h) * MD;
      const uint32_t st = lds0 + uint32_t((u % KSTAGES) * STAGE * 2);
      dma16_nt(src[k] + off, __builtin_amdgcn_readfirstlane(st + uint32_t(((8 * pw + k) * 4) * MD * 2)));
    };
    auto issue_k = [&](int u) __attribute__((always_inline)) {
#pragma unroll
      for (int k = 0; k < 8; ++k) issue_k_piece(u, k);
    };
    const uint16_t *msplit = reinterpret_cast<const uint16_t *>(base);
    const uint32_t mlds0 = lds0 + uint32_t(KSTAGES * STAGE * 2);
    const int npc = min(64, R16) >> 3;
    auto issue_m_piece = [&](int u, int k) __attribute__((always_inline)) {
      const uint16_t *m0 = msplit + int64_t(u) * R16 * 256;
      const uint32_t st = mlds0 + uint32_t((u & 1) * MSTAGE * 2);
      const int piece = pw * npc + k;
      const int r = piece * 2 + (lane >> 5);
      const int sl = lane & 31;
      dma16(m0 + r * 256 + ((sl ^ (r & 15)) * 8), __builtin_amdgcn_readfirstlane(st + uint32_t(piece * 1024)));
    };
    const int pp = 32 * pw + (lane & 31), hc = lane >> 5;
    float kb[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) kb[i] = 0.f;
    auto kbar_step = [&](const uint16_t *kr, int c) __attribute__((always_inline)) {
      const uint4 v = *reinterpret_cast<const uint4 *>(kr + (((8 * hc + c) ^ (pp & 15)) * 8));
      const uint32_t q[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        kb[8 * c + 2 * e] += __uint_as_float(q[e] << 16);
        kb[8 * c + 2 * e + 1] += __uint_as_float(q[e] & 0xffff0000u);
      }
    };
    // ---- producer 3: the owned rows. Lane l holds partials l + 64 q of the row (16 B each).
    // The loads into vv are inline assembly, invisible to the compiler's wait insertion:
    // from an o_issue until the wait that covers it nothing may touch vv's registers, so
    // every path that issues again (o_force) starts with no such load in flight.
    const bool owner = pw == 3;
    int oc = -1, orow = 0, onext = 0;
    u32x4 vv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) vv[q] = u32x4{0u, 0u, 0u, 0u};
    auto o_issue = [&](int x, int r) __attribute__((always_inline)) {
      const uint64_t *p = xpart + (int64_t(x) * R16 + r) * P * 2;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (lane + 64 * q < P) vv[q] = ld_coherent16(p + 2 * (lane + 64 * q));
    };
    auto o_landed = [&]() __attribute__((always_inline)) {   // order the reads of vv after a wait
#pragma unroll
      for (int q = 0; q < 8; ++q) asm volatile("" : "+v"(vv[q]));
    };
    auto o_finish = [&](int x, int r) __attribute__((always_inline)) -> bool {
      const uint64_t Sx = stamp + uint64_t(x);
      const uint32_t lo = uint32_t(Sx), hi = uint32_t(Sx >> 32);
      bool ok = true;
      float mx = -INFINITY;
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (lane + 64 * q < P) {
          ok = ok && vv[q].x == lo && vv[q].z == hi;
          mx = fmaxf(mx, __uint_as_float(vv[q].y));
        }
      if (!__all(ok)) return false;
      mx = wave_max(mx);
      float zs = 0.f;
      if (mx != -INFINITY)
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (lane + 64 * q < P) {
            const float mq = __uint_as_float(vv[q].y);
            if (mq != -INFINITY) zs += __uint_as_float(vv[q].w) * ex2(mq - mx);
          }
      zs = wave_sum(zs);
      const float c = (mx == -INFINITY || !(zs > 0.f)) ? -INFINITY : mx + log2f(zs);
      if (lane == 0) {
        uint64_t *o = xnrm + (int64_t(x) * R16 + r) * 2;
        st_word(o, c, lo);
        st_word(o + 1, c, hi);
      }
      return true;
    };
    // a row that must be finished now: retry until every partial is in (bounded)
    auto o_force = [&](int x, int r) __attribute__((always_inline)) {
      bool done = false;
      const uint32_t lim = timed_out ? 1u : spins;   // after one wait ran out, one try only
      for (uint32_t sp = 0; !done && sp < lim; ++sp) {
        if (sp) __builtin_amdgcn_s_sleep(2);
        o_issue(x, r);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        o_landed();
        done = o_finish(x, r);
      }
      if (!done) timed_out = true;
    };
    // the owned row of unit x, or -1
    auto o_row = [&](int x) __attribute__((always_inline)) {
      const int r = int((int64_t(wgi) - int64_t(x) * R16 % G + G) % G);
      return r < R ? r : -1;
    };

    issue_k(0);
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (k < npc) issue_m_piece(0, k);
    if (units > 1) issue_k(1);
    for (int u = 0; u < units; ++u) {
      if (u + 1 < units) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
      else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      fu_barrier();
      if (owner) {
        // the loads issued at the previous top are older than K(u + 1): they have landed
        o_landed();
        if (oc >= 0) {
          const bool done = o_finish(oc, orow);
          if (!done && oc + FU_LAG <= u) o_force(oc, orow);   // due: unit oc + 1 + FU_LAG needs it
          if (done || oc + FU_LAG <= u) oc = -1;
        }
        while (oc < 0 && onext <= u - 2) {                    // partials of unit u - 2 are out
          const int x = onext++;
          const int r = o_row(x);
          if (r >= 0) {
            oc = x;
            orow = r;
          }
        }
        if (oc >= 0) o_issue(oc, orow);
      }
      const uint16_t *kr = lds + (u % KSTAGES) * STAGE + pp * MD;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        if (c < 4) {
#pragma unroll
          for (int k = 2 * c; k < 2 * c + 2; ++k)
            if (k < npc && u + 1 < units) issue_m_piece(u + 1, k);
        } else if (u + 2 < units) {
          issue_k_piece(u + 2, 2 * (c - 4));
          issue_k_piece(u + 2, 2 * (c - 4) + 1);
        }
        if (KBAR) kbar_step(kr, c);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (owner) {
      // The loads of the last top may still be in flight, and the compiler's own wait
      // insertion does not see loads written in inline assembly: o_force would build its
      // addresses in vv's registers and a late return would overwrite them. Wait first.
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      o_landed();
      // the rows still open, in unit order, each waited for
      if (oc >= 0 && !o_finish(oc, orow)) o_force(oc, orow);
      for (int x = onext; x < units; ++x) {
        const int r = o_row(x);
        if (r >= 0) o_force(x, r);
      }
    }
    fu_barrier();                                    // the ring is free (matches the consumers)
    float *kt = reinterpret_cast<float *>(lds) + 2 * MFMA_TILE;
    constexpr int KT_ROW = MD + 4;
    if (KBAR) {
      const float inv = 1.0f / float(units);
#pragma unroll
      for (int q = 0; q < 16; ++q)
        *reinterpret_cast<float4 *>(kt + pp * KT_ROW + 64 * hc + 4 * q) =
            make_float4(kb[4 * q] * inv, kb[4 * q + 1] * inv, kb[4 * q + 2] * inv, kb[4 * q + 3] * inv);
    }
    fu_barrier();
    if (KBAR) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int pr = 32 * pw + 2 * q + (lane >> 5);
        const float4 v = *reinterpret_cast<const float4 *>(kt + pr * KT_ROW + 4 * (lane & 31));
        if (pr < ne) reinterpret_cast<float4 *>(base + z.off_kbar() + int64_t(pos_of(pr)) * MD)[lane & 31] = v;
      }
    }
    if (timed_out && host_fault) __hip_atomic_store(host_fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    return;
  }

  // ---------------- consumers
  const int rh = w & 1, ph = w >> 1, p0 = 64 * ph;
  const int jr = lane & 31, hl = lane >> 5;
  const int mrow = 32 * rh + jr;                    // this lane's memory row
  const bool real_row = mrow < R;
  // LDS: key entry p0 + 32 t + jr (16-byte chunk slots swizzled by jr & 15) and the split
  // memory row (channel block cb at chunk ((cb % 4) * 4 + cb / 4) * 2, then lo, swizzled)
  // the entry (within the tile) of slot value v of block t, and of the lane's scattered sum
  auto entry_of = [&](int tb, int v) __attribute__((always_inline)) { return p0 + 32 * tb + 8 * (v >> 2) + 4 * hl + (v & 3); };
  const int my_a = lane & 31;
  const int my_entry = entry_of(my_a >> 4, my_a & 15);
  // bit a of vmask: slot value a (block a / 16, value a % 16) is an entry of the tile
  uint32_t vmask = 0u;
#pragma unroll
  for (int a = 0; a < 32; ++a) vmask |= uint32_t(entry_of(a >> 4, a & 15) < ne) << a;
  f32x16 X[FU_SLOTS][2];
  float mh[FU_SLOTS];
#pragma unroll
  for (int i = 0; i < FU_SLOTS; ++i) {
    X[i][0] = f32x16{};
    X[i][1] = f32x16{};
    mh[i] = -INFINITY;
  }
  float pos_acc = 0.f;
  uint64_t pre0 = 0, pre1 = 0;                       // normaliser words of the next unit to finish
  auto prefetch = [&](int x) __attribute__((always_inline)) {
    if (real_row) {
      const uint64_t *p = xnrm + (int64_t(x) * R16 + mrow) * 2;
      pre0 = ld_word(p);
      pre1 = ld_word(p + 1);
    }
  };
  // finish unit x: weight its rows by exp2(m - c), sum over the rows (reduce-scatter)
  auto fin = [&](int x, f32x16 (&E)[2], float m) __attribute__((always_inline)) {
    const uint64_t Sx = stamp + uint64_t(x);
    const uint32_t lo = uint32_t(Sx), hi = uint32_t(Sx >> 32);
    const bool need = real_row && m != -INFINITY;
    uint64_t a = pre0, b = pre1;
    auto ready = [&]() __attribute__((always_inline)) { return uint32_t(a) == lo && uint32_t(b) == hi; };
    uint32_t sp = 0;
    const uint32_t lim = timed_out ? 0u : spins;     // after one wait ran out, no more waiting
    while (!__all(!need || ready()) && sp < lim) {
      __builtin_amdgcn_s_sleep(1);
      if (need && !ready()) {
        const uint64_t *p = xnrm + (int64_t(x) * R16 + mrow) * 2;
        a = ld_word(p);
        b = ld_word(p + 1);
      }
      ++sp;
    }
    if (!__all(!need || ready())) timed_out = true;
    const float c = __uint_as_float(uint32_t(a >> 32));
    const float f = need && ready() && c != -INFINITY ? ex2(m - c) : 0.f;
    // a row that takes no part adds an exact zero (a pad row's logits come from stale LDS)
    const bool add = need && f != 0.f;
    float r[32];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      r[q] = add ? f * E[0][q] : 0.f;
      r[16 + q] = add ? f * E[1][q] : 0.f;
    }
    // reduce-scatter over the 32 lanes of the half: in the step on bit b the lane keeps the
    // indices whose bit b equals its own and adds a partner's, a lane with the other bit b
    // and the same higher bits (lane ^ 16, then within a row its mirror, half-row mirror,
    // quad mirror and quad neighbour: DPP moves). The lane ends with index lane % 32.
    int lb = lane;
    asm volatile("" : "+v"(lb));
    auto rs_step = [&](auto mov, int sb) __attribute__((always_inline)) {
      const bool up = (lb & sb) != 0;
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (q < sb) {
          const float keep = up ? r[q + sb] : r[q];
          const float give = up ? r[q] : r[q + sb];
          r[q] = keep + mov(give);
        }
    };
    rs_step([&](float x) __attribute__((always_inline)) { return __shfl_xor(x, 16, WAVE); }, 16);
    rs_step([](float x) __attribute__((always_inline)) { return dpp_mov<0x140>(x); }, 8);   // row_mirror
    rs_step([](float x) __attribute__((always_inline)) { return dpp_mov<0x141>(x); }, 4);   // row_half_mirror
    rs_step([](float x) __attribute__((always_inline)) { return dpp_mov<0x1B>(x); }, 2);    // quad_perm [3,2,1,0]
    rs_step([](float x) __attribute__((always_inline)) { return dpp_mov<0xB1>(x); }, 1);    // quad_perm [1,0,3,2]
    pos_acc += r[0];
  };
  auto stats_store = [&](int x, float m, float zsum) __attribute__((always_inline)) {
    if (hl == 0 && real_row) {
      const uint64_t Sx = stamp + uint64_t(x);
      uint64_t *o = xpart + ((int64_t(x) * R16 + mrow) * P + 2 * wgi + ph) * 2;
      st_word(o, m, uint32_t(Sx));
      st_word(o + 1, zsum, uint32_t(Sx >> 32));
    }
  };
  // the last unit's row statistics, without MFMAs to hide them under
  auto last_stats = [&](f32x16 (&E)[2], float &mo) __attribute__((always_inline)) {
    float m = -INFINITY, zsum = 0.f;
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        if (!((vmask >> (16 * tb + q)) & 1u)) E[tb][q] = -INFINITY;
        m = fmaxf(m, E[tb][q]);
      }
    m = fmaxf(m, __shfl_xor(m, 32, WAVE));
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        E[tb][q] = m == -INFINITY ? 0.f : ex2(E[tb][q] - m);
        zsum += E[tb][q];
      }
    zsum += __shfl_xor(zsum, 32, WAVE);
    mo = m;
    stats_store(units - 1, m, zsum);
  };
  // unit v's MFMAs into C, with unit v - 1's row statistics (slot E, max mo) folded in
  // Steps past the last unit (v >= units) run no MFMAs: step `units` takes the last unit's
  // statistics, and the steps up to units + FU_LAG finish the units still open.
  auto step = [&](int v, f32x16 (&C)[2], float &mc, f32x16 (&E)[2], float &mo) __attribute__((always_inline)) {
    if (v - 1 - FU_LAG >= 0 && v - 1 - FU_LAG < units) fin(v - 1 - FU_LAG, C, mc);
    if (v - FU_LAG >= 0 && v - FU_LAG < units) prefetch(v - FU_LAG);
    if (v >= units) {
      if (v == units) last_stats(E, mo);
      return;
    }
    fu_barrier();                                    // stage v in LDS
    const bool epi = v >= 1;
    // lane constants re-derived in every step: hoisted out of the unit loop they would
    // stay live across it (address offsets per k-step, the entry mask)
    int lx = lane;
    asm volatile("" : "+v"(lx));
    uint32_t vm = vmask;
    asm volatile("" : "+v"(vm));
    const int ljr = lx & 31, lhl = lx >> 5, lsw = lx & 15, lrow = 32 * rh + ljr;
    const uint16_t *kl = lds + (v % KSTAGES) * STAGE + (p0 + ljr) * MD;
    const uint16_t *mb = lds + KSTAGES * STAGE + (v & 1) * MSTAGE + lrow * 256;
    bf16x8 ka0[2], ka1[2], mhi[2], mlo[2];
    auto read_ks = [&](int ks, int bsel) __attribute__((always_inline)) {
      const int cb = 2 * ks + lhl;
      const int ko = (cb ^ lsw) * 8;
      const int mc = (((cb & 3) * 4 + (cb >> 2)) * 2) ^ lsw;
      ka0[bsel] = *reinterpret_cast<const bf16x8 *>(kl + ko);
      ka1[bsel] = *reinterpret_cast<const bf16x8 *>(kl + 32 * MD + ko);
      mhi[bsel] = *reinterpret_cast<const bf16x8 *>(mb + mc * 8);
      mlo[bsel] = *reinterpret_cast<const bf16x8 *>(mb + (mc ^ 1) * 8);
    };
    C[0] = f32x16{};
    C[1] = f32x16{};
    read_ks(0, 0);
    float m = -INFINITY, zsum = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const int bs = ks & 1;
      if (ks + 1 < 8) read_ks(ks + 1, bs ^ 1);
      C[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka0[bs], mhi[bs], C[0], 0, 0, 0);
      C[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka1[bs], mhi[bs], C[1], 0, 0, 0);
      C[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka0[bs], mlo[bs], C[0], 0, 0, 0);
      C[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka1[bs], mlo[bs], C[1], 0, 0, 0);
      if (epi) {
        if (ks < 2) {                                 // block ks: mask past the tile, row maximum
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            if (!((vm >> (16 * ks + q)) & 1u)) E[ks][q] = -INFINITY;
            m = fmaxf(m, E[ks][q]);
          }
          if (ks == 1) m = fmaxf(m, __shfl_xor(m, 32, WAVE));
        } else if (ks < 6) {                          // exp2 of eight values
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const int a = 8 * (ks - 2) + q, tb = a >> 4, qq = a & 15;
            E[tb][qq] = m == -INFINITY ? 0.f : ex2(E[tb][qq] - m);
          }
        } else if (ks == 6) {
#pragma unroll
          for (int q = 0; q < 16; ++q) zsum += E[0][q] + E[1][q];
          zsum += __shfl_xor(zsum, 32, WAVE);
        } else {
          mo = m;
          stats_store(v - 1, m, zsum);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  for (int v0 = 0; v0 <= units + FU_LAG; v0 += FU_SLOTS) {
    step(v0, X[0], mh[0], X[4], mh[4]);
    step(v0 + 1, X[1], mh[1], X[0], mh[0]);
    step(v0 + 2, X[2], mh[2], X[1], mh[1]);
    step(v0 + 3, X[3], mh[3], X[2], mh[2]);
    step(v0 + 4, X[4], mh[4], X[3], mh[3]);
  }
  fu_barrier();                                      // the ring is free: reuse it for the reduction
  float *red = reinterpret_cast<float *>(lds);       // [2][MFMA_TILE]
  red[rh * MFMA_TILE + my_entry] = pos_acc;
  fu_barrier();
  if (t < ne) scores[s.slot_off + pos_of(t)] = red[t] + red[MFMA_TILE + t];
  if (timed_out && host_fault) __hip_atomic_store(host_fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// ------------------------------------------------------------------ first pass, unit-major (R <= 64, even Hkv)
// The first pass needs no sum over units per position, so it runs unit by unit: a
// workgroup owns one head pair of one layer and a chunk of CH positions. The memory
// rows of its two units sit in registers for the whole chunk and only keys stream,
// 32 positions x 2 heads (16 KB) per stage through a 4-stage LDS ring, so two
// workgroups share a CU. Wave w takes head w >> 1 of the pair and memory rows
// 32 (w & 1) .. + 31 as two 16-row MFMA blocks; per row it keeps an online (max, sum
// of exp2) over the chunk's candidates and writes one partial per (chunk, unit, row).
// Non-candidates enter the accumulators as -inf before the MFMAs, so the epilogue
// needs no mask. The memory rows are read as float32 and split in registers; the
// workgroups of chunk 0 also store the split rows of their units for the second pass
// and, with the residual head on, the column sums of their rows (a partial of mbar).
// For a session at or under its budget the pass only fills the scores with -inf.
constexpr int ST_TILE = 32;                      // positions per stage
constexpr int ST_STAGE = ST_TILE * 2 * MD;       // bf16 per stage: 32 positions x 2 heads
constexpr int ST_CHMAX = 1024;                   // positions per chunk at most


// 16 bytes per lane from sbase + voff (scalar base, 32-bit byte offset per lane)
// straight into LDS at lds_base + 16 * lane, with the non-temporal hint of the key
// streams (dma16_nt).
__device__ __forceinline__ void dma16s(const void *sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
               :
               : "s"(lds_base), "v"(voff), "s"(sbase)
               : "memory", "m0");
}

// NW waves per head, each holding 32 rows: 2 for sessions of up to 64 memory rows
// (256 threads, two waves per SIMD), 4 for up to 128 (512 threads, four waves per
// SIMD); either way two workgroups share a CU. A batch that holds both kinds of
// session runs one launch of each, and each launch skips the other's sessions
// (`big`: 0 every session, 1 only R <= 64, 2 only R > 64).
//
// MASS: the same pass after the row normalisers are known (the SnapKV-style scorer):
// the accumulators start from the rows' seeds -(max + log2 Z), so exp2 of a logit is
// its softmax weight, and each position keeps its attention mass in this unit (the
// sum over the unit's rows) instead of the rows' statistics. The masses of a tile are
// summed over the waves of a head through a small LDS buffer at the top of the next
// tile and parked in the tile's bias / key-offset entries, which no later step reads;
// the chunk's masses leave once, at the end: umass[u][slot_off + j] (row stride
// ustride), zero off the candidates.
template <int NW, bool MASS = false>
__global__ void __launch_bounds__(128 * NW) __attribute__((amdgpu_waves_per_eu(NW, NW)))
k_score_stats(const uint16_t *__restrict__ kpool, int64_t num_slots, int L, int Hkv, int dead,
              const ikv_session *__restrict__ sess, const int32_t *__restrict__ slot_maps, float *__restrict__ ws,
              const float *__restrict__ M, float *__restrict__ scores, bool resid, int CH, int big,
              float *__restrict__ umass = nullptr, int64_t ustride = 0) {
  constexpr int ST_THREADS = 128 * NW;
  constexpr int ST_STAGES = 4;
  constexpr int KI = 8 / NW;                     // key loads (1 KB each) per wave per stage
  __shared__ __align__(1024) uint16_t ring[ST_STAGES * ST_STAGE];
  __shared__ uint32_t koff[ST_CHMAX];            // byte offset of each position's key rows in the layer
  __shared__ __align__(16) float bias[ST_CHMAX];  // 0 for a candidate, -inf otherwise
  __shared__ float mred[MASS ? 2 * 2 * NW * ST_TILE : 1];   // per tile parity, head, wave: 32 masses

  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if ((big == 1 && s.R > 64) || (big == 2 && s.R <= 64)) return;   // the other launch's session
  const int HP = L * Hkv / 2;
  const int hp = int(blockIdx.x % unsigned(HP)), chunk = int(blockIdx.x / unsigned(HP));
  const int c0 = chunk * CH;
  if (c0 >= s.N) return;
  if (s.N <= s.C) {                              // the gate: nothing is scored
    if (hp == 0 && !MASS)
      for (int j = c0 + int(threadIdx.x); j < min(s.N, c0 + CH); j += ST_THREADS) scores[s.slot_off + j] = -INFINITY;
    return;
  }
  // the chunk's entries: its candidates from the list (MASS: every position of the chunk)
  const ScoreSizes z0 = score_sizes(s, L, L * Hkv, MD, resid, true);
  const float *wsb = ws + score_offset(sess, b, L, L * Hkv, MD, resid, true);
  const int32_t *lst = reinterpret_cast<const int32_t *>(wsb + z0.off_clist());
  const int npos = MASS ? min(CH, s.N - c0) : reinterpret_cast<const int32_t *>(wsb + z0.off_ccount(s.N))[chunk];
  const bool ident = MASS || npos == min(CH, s.N - c0);   // every position a candidate: its own list
  const int T = int(cdiv(npos, ST_TILE));
  const int l = hp / (Hkv / 2), h0 = 2 * (hp - l * (Hkv / 2));
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int hh = w / NW, r0 = 32 * (w % NW);     // head within the pair, first memory row
  const int g = lane >> 4, r16 = lane & 15;
  const int R = s.R;
  const int units = L * Hkv;
  const int u = l * Hkv + h0 + hh;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  uint16_t *msplit = reinterpret_cast<uint16_t *>(base);
  float *part = base + z.off_part();
  const int32_t *S = slot_maps + s.slot_off;
  const uint32_t slot_bytes = uint32_t(Hkv) * MD * 2;

  // the chunk's key offsets (dead slot past the end) and candidate biases
  int32_t sv[ST_CHMAX / ST_THREADS];
#pragma unroll
  for (int k = 0; k < ST_CHMAX / ST_THREADS; ++k) {
    const int p = t + k * ST_THREADS;
    sv[k] = p < npos ? S[ident ? c0 + p : lst[c0 + p]] : dead;
  }
  // memory rows of this wave as B-operand fragments: lane (g, r16) holds row r0 + 16 rb + r16
  // (the last row stands in for rows past R, whose results are never stored), channels
  // (4 ks + g) * 8 .. + 8 of M * log2(e) / sqrt(D), split into bf16 hi + lo (both rounded
  // to nearest even)
  bf16x8 mh[2][4], ml[2][4];
  {
    const float mscale = LOG2E / sqrtf(float(MD));
    float4 mv[2][4][2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int row = min(r0 + 16 * rb + r16, R - 1);
      const float *mp = M + s.mem_off + (int64_t(u) * R + row) * MD + g * 8;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        mv[rb][ks][0] = *reinterpret_cast<const float4 *>(mp + ks * 32);
        mv[rb][ks][1] = *reinterpret_cast<const float4 *>(mp + ks * 32 + 4);
      }
    }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const float x[8] = {mv[rb][ks][0].x, mv[rb][ks][0].y, mv[rb][ks][0].z, mv[rb][ks][0].w,
                            mv[rb][ks][1].x, mv[rb][ks][1].y, mv[rb][ks][1].z, mv[rb][ks][1].w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float v = x[e] * mscale;
          mh[rb][ks][e] = __bf16(v);
          ml[rb][ks][e] = __bf16(v - float(mh[rb][ks][e]));
        }
      }
    // chunk 0 keeps the split rows for the second pass, in the layout of k_msplit (rows
    // padded to whole slices, the pad rows zero)
    if (chunk == 0 && !MASS)
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const int row = r0 + 16 * rb + r16;
        if (row < pad16(R)) {
          uint16_t *dp = msplit + (int64_t(u) * pad16(R) + row) * 256;
          const bool real = row < R;
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
            *reinterpret_cast<bf16x8 *>(dp + (g * 4 + ks) * 16) = real ? mh[rb][ks] : bf16x8{};
            *reinterpret_cast<bf16x8 *>(dp + (g * 4 + ks) * 16 + 8) = real ? ml[rb][ks] : bf16x8{};
          }
        }
      }
  }
#pragma unroll
  for (int k = 0; k < ST_CHMAX / ST_THREADS; ++k) {
    const int p = t + k * ST_THREADS, j = c0 + p;
    const bool in = p < npos;
    const int slot = in ? sv[k] : dead;
    // list entries are candidates; the mass pass walks positions and tests them
    const bool cand = in && (!MASS || (slot != dead && !(j < s.pi || (j >= s.qs && j < s.qe))));
    koff[p] = uint32_t(slot) * slot_bytes;
    bias[p] = cand ? 0.f : -INFINITY;
  }
  // the mass pass: seeds of the lane's two rows (-inf past R, so those rows add nothing)
  float sd[2] = {0.f, 0.f};
  if constexpr (MASS) {
    const float *nl2 = base + z.off_nl2();
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int row = r0 + 16 * rb + r16;
      sd[rb] = row < R ? nl2[int64_t(u) * R + row] : -INFINITY;
    }
  }
  // every compiler-issued load of the set-up is complete before the first key load
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // Key loads: instruction k of wave w fills 1 KB of the stage, positions 2 (KI w + k)
  // and + 1; lane -> (position, head, 16-byte slot lane & 15), and slot s of a 256-byte
  // row holds chunk s ^ (position & 15).
  const uint16_t *kb0 = kpool + int64_t(l) * num_slots * (int64_t(Hkv) * MD) + int64_t(h0) * MD;
  uint32_t lconst[KI];
#pragma unroll
  for (int k = 0; k < KI; ++k) {
    const int p = 2 * (KI * w + k) + (lane >> 5);
    lconst[k] = uint32_t(((lane >> 4) & 1) * MD * 2 + (((lane & 15) ^ (p & 15)) * 16));
  }
  const uint32_t lds_w =
      __builtin_amdgcn_readfirstlane(uint32_t(reinterpret_cast<uintptr_t>(ring)) + w * KI * 1024);
  auto issue = [&](int tt) {
    const uint32_t st = lds_w + uint32_t((tt % ST_STAGES) * ST_STAGE * 2);
#pragma unroll
    for (int k = 0; k < KI; ++k)
      dma16s(kb0, koff[tt * ST_TILE + 2 * (KI * w + k) + (lane >> 5)] + lconst[k], st + k * 1024);
  };

  float Mr[2] = {-INFINITY, -INFINITY}, Zr[2] = {0.f, 0.f};
  auto compute = [&](int tt) {
    const uint16_t *kl = ring + (tt % ST_STAGES) * ST_STAGE;
    bf16x8 ka[2][4];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const uint16_t *kr = kl + ((16 * pb + r16) * 2 + hh) * MD;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) ka[pb][ks] = *reinterpret_cast<const bf16x8 *>(kr + (((4 * ks + g) ^ r16) * 8));
    }
    // lane (g, r16) of block (pb, rb) holds row r0 + 16 rb + r16 at positions 16 pb + 4 g + i
    f32x4 acc[2][2];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const float4 bv = *reinterpret_cast<const float4 *>(bias + tt * ST_TILE + 16 * pb + 4 * g);
      acc[pb][0] = f32x4{bv.x + sd[0], bv.y + sd[0], bv.z + sd[0], bv.w + sd[0]};
      acc[pb][1] = f32x4{bv.x + sd[1], bv.y + sd[1], bv.z + sd[1], bv.w + sd[1]};
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          acc[pb][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[pb][ks], mh[rb][ks], acc[pb][rb], 0, 0, 0);
          acc[pb][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[pb][ks], ml[rb][ks], acc[pb][rb], 0, 0, 0);
        }
    if constexpr (MASS) {
      // position 16 pb + 4 g + i: its softmax weights under the wave's 32 rows, summed
      // over the 16 lanes of the lane group
      float pm[2][4];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pm[pb][i] = row16_sum(ex2(acc[pb][0][i]) + ex2(acc[pb][1][i]));
        }
      if (r16 == 0) {
        float *mr = mred + (((tt & 1) * 2 + hh) * NW + (w % NW)) * ST_TILE;
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int i = 0; i < 4; ++i) mr[16 * pb + 4 * g + i] = pm[pb][i];
      }
      return;
    }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float m = Mr[rb];
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int i = 0; i < 4; ++i) m = fmaxf(m, acc[pb][rb][i]);
      const float e0 = (m == -INFINITY) ? 0.f : m;   // nothing seen yet: every term below is 0
      float zs = Zr[rb] * ex2(Mr[rb] - e0);
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int i = 0; i < 4; ++i) zs += ex2(acc[pb][rb][i] - e0);
      Zr[rb] = zs;
      Mr[rb] = m;
    }
  };

  const bool act = __builtin_amdgcn_readfirstlane(r0) < R;   // a wave past the last row only loads
  // the mass pass: tile k's masses of head hh, summed over the head's active waves (in
  // wave order), into bias (head 0) or koff (head 1) at the tile's positions
  auto mass_fold = [&](int k) {
    if (!MASS || w % NW != 0 || lane >= ST_TILE) return;
    const int nwa = min(NW, (R + 31) / 32);
    const float *mr = mred + ((k & 1) * 2 + hh) * NW * ST_TILE + lane;
    float v = 0.f;
    for (int q = 0; q < nwa; ++q) v += mr[q * ST_TILE];
    if (hh == 0) bias[k * ST_TILE + lane] = v;
    else koff[k * ST_TILE + lane] = __float_as_uint(v);
  };
  for (int k = 0; k < ST_STAGES - 1 && k < T; ++k) issue(k);
  for (int tt = 0; tt < T; ++tt) {
    // tile tt's KI loads per wave are done once at most those of the later tiles
    // already issued (KI each) are outstanding
    vm_wait(KI * min(ST_STAGES - 2, T - 1 - tt));
    __syncthreads();
    if (tt + ST_STAGES - 1 < T) issue(tt + ST_STAGES - 1);
    if (tt > 0) mass_fold(tt - 1);
    if (act) compute(tt);
  }
  if constexpr (MASS) {
    __syncthreads();
    mass_fold(T - 1);
    __syncthreads();
    const int u0 = l * Hkv + h0;
    float *o0 = umass + int64_t(u0) * ustride + s.slot_off + c0, *o1 = o0 + ustride;
    for (int p = t; p < npos; p += ST_THREADS) {
      o0[p] = bias[p];
      o1[p] = __uint_as_float(koff[p]);
    }
    return;
  }

  // chunk 0 with the residual head: column sums of the head pair's 2 R memory rows
  if (resid && chunk == 0) {
    float *red = reinterpret_cast<float *>(ring);  // the ring is free: every wave is past its last tile
    __syncthreads();
    constexpr int NP = ST_THREADS / MD;          // row classes summed apart, then in order
    const int c = t & (MD - 1), part = t / MD;
    const float *mp = M + s.mem_off + int64_t(l * Hkv + h0) * R * MD + c;
    float a = 0.f;
    for (int r = part; r < 2 * R; r += NP) a += mp[int64_t(r) * MD];
    red[t] = a;
    __syncthreads();
    if (t < MD) {
      float tot = 0.f;
#pragma unroll
      for (int q = 0; q < NP; ++q) tot += red[q * MD + t];
      base[z.off_mbp() + int64_t(hp) * MD + t] = tot;
    }
  }

  // merge the four lane groups of each row and store the chunk's partial
  const int64_t rows = int64_t(units) * R;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
    for (int o = 16; o < 64; o <<= 1) {
      const float m2 = __shfl_xor(Mr[rb], o, WAVE), z2 = __shfl_xor(Zr[rb], o, WAVE);
      const float mm = fmaxf(Mr[rb], m2);
      const float x = (Mr[rb] == -INFINITY) ? 0.f : Zr[rb] * ex2(Mr[rb] - mm);
      const float y = (m2 == -INFINITY) ? 0.f : z2 * ex2(m2 - mm);
      Mr[rb] = mm;
      Zr[rb] = x + y;
    }
    const int row = r0 + 16 * rb + r16;
    if (g == 0 && row < R)
      *reinterpret_cast<float2 *>(part + (int64_t(chunk) * rows + int64_t(u) * R + row) * 2) = make_float2(Mr[rb], Zr[rb]);
  }
}

// Per (unit, row): combine the per-tile statistics into (max, 1/Z), log2 domain.
// A workgroup takes 64 consecutive rows; its eight waves split the tiles (lane =
// row, so each load instruction reads 512 contiguous bytes), fold them online into
// (max, sum) and merge through LDS in a fixed order. With the residual head on, the
// first workgroups of each session do the head's set-up instead, which needs only the
// first pass: with `kv` (the matrix-core head) RES_KEYS workgroups build K' and V' of
// one live query row each from the keys (res_kv_keys_wg) and `nfold` fold the first
// layer (res_fold_wg), then one workgroup writes mbar and the live query positions
// (res_setup_body).
__global__ void __launch_bounds__(512) k_lse_mfma(const ikv_session *__restrict__ sess, float *__restrict__ ws, int L,
                                                  int Hkv, bool resid, int ptile, int pper,
                                                  const int32_t *__restrict__ slot_maps,
                                                  const int32_t *__restrict__ qpos, int dead, bool pairs, bool kv,
                                                  int nfold, const uint16_t *__restrict__ kpool, int64_t num_slots,
                                                  const float *__restrict__ blob, float *__restrict__ shared) {
  __shared__ float sm[8][64], sz[8][64];
  const int b = blockIdx.y;
  const int nkv = kv ? RES_KEYS : 0;
  const int extra = resid ? nkv + nfold + 1 : 0;
  const int bx = int(blockIdx.x) - extra;
  if (bx < 0) {
    const int x = int(blockIdx.x);
    if (x < nkv)
      res_kv_keys_wg<MD>(x, sess, b, kpool, num_slots, L, Hkv, slot_maps, qpos, dead, blob, ws);
    else if (x < nkv + nfold)
      res_fold_wg<MD>(x - nkv, sess, b, blob, ws, shared, L, Hkv, pairs);
    else
      res_setup_body<MD>(sess, b, slot_maps, qpos, dead, ws, L, Hkv, true, pairs);
    return;
  }
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  const int units = L * Hkv;
  const int64_t rows = int64_t(units) * s.R;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t i = int64_t(bx) * 64 + lane;
  if (int64_t(bx) * 64 >= rows) return;
  const bool on = i < rows;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const float *part = base + z.off_part();
  // partials: one per ptile positions, or pper per ptile-position chunk (list tiles)
  const int64_t tiles = pper > 0 ? cdiv(s.N, ptile) * pper : cdiv(s.N, ptile);
  float m = -INFINITY, zs = 0.f;
  constexpr int LB = 8;                            // tiles in flight per thread
  if (on)
    for (int64_t k0 = w; k0 < tiles; k0 += 8 * LB) {
      float2 pv[LB];
#pragma unroll
      for (int q = 0; q < LB; ++q) {
        const int64_t k = k0 + 8 * q;
        pv[q] = *reinterpret_cast<const float2 *>(part + (min(k, tiles - 1) * rows + i) * 2);
        if (k >= tiles) pv[q] = make_float2(-INFINITY, 0.f);
      }
#pragma unroll
      for (int q = 0; q < LB; ++q) {
        const float2 p = pv[q];
        if (p.x == -INFINITY) continue;
        if (p.x > m) {
          zs = (m == -INFINITY ? 0.f : zs * exp2f(m - p.x)) + p.y;
          m = p.x;
        } else {
          zs += p.y * exp2f(p.x - m);
        }
      }
    }
  sm[w][lane] = m;
  sz[w][lane] = zs;
  __syncthreads();
  if (w == 0 && on) {
    float mx = -INFINITY;
    for (int k = 0; k < 8; ++k) mx = fmaxf(mx, sm[k][lane]);
    double Z = 0.0;
    if (mx != -INFINITY)
      for (int k = 0; k < 8; ++k)
        if (sm[k][lane] != -INFINITY) Z += double(sz[k][lane]) * double(exp2f(sm[k][lane] - mx));
    float *lse = base + z.off_lse();
    lse[2 * i] = mx;
    lse[2 * i + 1] = Z > 0.0 ? float(1.0 / Z) : 0.f;
    // -(max + log2 Z): the second pass seeds its accumulators with it (-inf without candidates)
    float *nl2 = base + z.off_nl2();
    nl2[i] = (mx == -INFINITY || !(Z > 0.0)) ? -INFINITY : float(-(double(mx) + log2(Z)));
  }
}

// The candidate list of each session for the MFMA passes: chunk c (CH positions)
// keeps its candidates in position order at clist[c CH ...] and their count at
// ccount[c]; every other position's score is -inf (all of them for a session at or
// under its budget, whose counts are zero). One workgroup per (chunk, session); the
// order within a chunk comes from wave ballots and a prefix over the waves.
constexpr int CLIST_THREADS = 1024;              // a whole chunk (at most 1024 positions) per round

__global__ void __launch_bounds__(CLIST_THREADS) k_cand_list(const ikv_session *__restrict__ sess,
                                                             const int32_t *__restrict__ slot_maps, int dead,
                                                             float *__restrict__ ws, float *__restrict__ scores,
                                                             int L, int Hkv, bool resid, int CH) {
  __shared__ int wsum[CLIST_THREADS / WAVE];
  const int b = blockIdx.y, c = blockIdx.x;
  const ikv_session s = sess[b];
  const int c0 = c * CH;
  if (c0 >= s.N) return;
  const int units = L * Hkv;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  int32_t *lst = reinterpret_cast<int32_t *>(base + z.off_clist()) + c0;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const bool gated = s.N <= s.C;
  int count = 0;
  for (int r = 0; r < CH; r += CLIST_THREADS) {
    const int j = c0 + r + t;
    const bool in = r + t < CH && j < s.N;         // a round may reach past a 128-position chunk
    const bool cand = in && !gated && slot_maps[s.slot_off + j] != dead && !(j < s.pi || (j >= s.qs && j < s.qe));
    if (in && !cand) scores[s.slot_off + j] = -INFINITY;
    const uint64_t m = __ballot(cand);
    if (lane == 0) wsum[w] = __popcll(m);
    __syncthreads();
    int off = count;
    for (int q = 0; q < w; ++q) off += wsum[q];
    if (cand) lst[off + __popcll(m & ((uint64_t(1) << lane) - 1))] = j;
    for (int q = 0; q < CLIST_THREADS / WAVE; ++q) count += wsum[q];
    __syncthreads();
  }
  if (t == 0) reinterpret_cast<int32_t *>(base + z.off_ccount(s.N))[c] = count;
}

// The one-key-pass form's rule score: per list entry, the sum over units and rows of
// exp2(logit + seed), seed = -(max + log2 Z) of the row (Eq. 3), from the stash. A
// workgroup owns one 128-entry list tile; thread (group, quad) adds entries 4 quad .. + 3
// of every 16th (unit, row), four in one 16-byte load, and the 16 groups are added in
// group order through LDS.
constexpr int SS_THREADS = 512;

__global__ void __launch_bounds__(SS_THREADS) k_score_stash(const ikv_session *__restrict__ sess,
                                                            const int32_t *__restrict__ slot_maps,
                                                            const float *__restrict__ ws, float *__restrict__ scores,
                                                            int L, int Hkv, bool resid, int CH) {
  __shared__ float red[SS_THREADS / 32][MFMA_TILE];
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;
  // list tiles in the grid order of k_score_ws (tile-index-major)
  const int per = CH / MFMA_TILE, nch = int(gridDim.x) / per;
  const int lc = int(blockIdx.x) % nch, lk = int(blockIdx.x) / nch;
  if (int64_t(lc) * CH >= s.N) return;
  const int units = L * Hkv;
  const ScoreSizes z = score_sizes(s, L, units, MD, resid, true);
  const float *base = ws + score_offset(sess, b, L, units, MD, resid, true);
  const int cnt = reinterpret_cast<const int32_t *>(base + z.off_ccount(s.N))[lc];
  const int ne = min(MFMA_TILE, cnt - lk * MFMA_TILE);
  if (ne <= 0) return;
  const int32_t *lst = reinterpret_cast<const int32_t *>(base + z.off_clist()) + lc * CH + lk * MFMA_TILE;
  const bool ident = cnt == min(CH, s.N - lc * CH);
  const int e0 = lc * CH + lk * MFMA_TILE;
  const int t = threadIdx.x, q = t & 31, grp = t >> 5;
  const int64_t NS = stash_stride(s.N);
  const float *st = base + z.off_stash() + e0 + 4 * q;
  const float *nl2 = base + z.off_nl2();
  const int rows = units * s.R;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  constexpr int UN = 8;                              // (unit, row) loads in flight per thread
  for (int i0 = grp; i0 < rows; i0 += 16 * UN) {
    float4 v[UN];
    float sd[UN];
#pragma unroll
    for (int k = 0; k < UN; ++k) {
      const int i = min(i0 + 16 * k, rows - 1);
      const f32x4 x = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(st + int64_t(i) * NS));
      v[k] = make_float4(x[0], x[1], x[2], x[3]);
      sd[k] = i0 + 16 * k < rows ? nl2[i] : -INFINITY;   // past the last row: adds nothing
    }
#pragma unroll
    for (int k = 0; k < UN; ++k) {
      a.x += ex2(v[k].x + sd[k]);
      a.y += ex2(v[k].y + sd[k]);
      a.z += ex2(v[k].z + sd[k]);
      a.w += ex2(v[k].w + sd[k]);
    }
  }
  *reinterpret_cast<float4 *>(&red[grp][4 * q]) = a;
  __syncthreads();
  if (t < ne) {
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < SS_THREADS / 32; ++k) v += red[k][t];
    scores[s.slot_off + (ident ? e0 + t : lst[t])] = v;   // every list entry is a candidate
  }
}

// The SnapKV-style score: for each candidate j, the sum over units u of the largest
// attention mass among positions j - 3 .. j + 3 of unit u (a max pool of 7 positions,
// positions outside [0, N) left out; non-candidates hold zero mass). A workgroup owns 64
// positions; its four waves take every fourth unit, each lane one position, and their
// sums are added in wave order.
constexpr int PL_POS = 64;

__global__ void __launch_bounds__(256) k_pool7(const ikv_session *__restrict__ sess,
                                               const int32_t *__restrict__ slot_maps, int dead,
                                               const float *__restrict__ umass, int64_t ustride, int units,
                                               float *__restrict__ scores) {
  __shared__ float part[4][PL_POS];
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  if (s.N <= s.C) return;                          // the gate: the first pass wrote -inf
  const int j0 = blockIdx.x * PL_POS;
  if (j0 >= s.N) return;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int j = j0 + lane;
  const int jj = min(j, s.N - 1);
  int nb[7];
#pragma unroll
  for (int d = 0; d < 7; ++d) nb[d] = min(max(jj + d - 3, 0), s.N - 1);   // clamped: repeats leave the max alone
  const float *base = umass + s.slot_off;
  float acc = 0.f;
  for (int u = w; u < units; u += 4) {
    const float *v = base + int64_t(u) * ustride;
    float m = v[nb[0]];
#pragma unroll
    for (int d = 1; d < 7; ++d) m = fmaxf(m, v[nb[d]]);
    acc += m;
  }
  part[w][lane] = acc;
  __syncthreads();
  if (w == 0 && j < s.N) {
    const int32_t slot = slot_maps[s.slot_off + j];
    const bool c = slot != dead && !(j < s.pi || (j >= s.qs && j < s.qe));
    scores[s.slot_off + j] = c ? ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane] : -INFINITY;
  }
}

hipError_t launch_residual(const ScoreArgs &a, hipStream_t st);

// ---- the one-key-pass form at R <= 64 (k_score_fused): when it applies, and its exchange area
namespace {

// Workgroups a cooperative launch of k_score_fused may hold on the current device (0: none).
int fused_capacity() {
  static int cap[64];
  static bool known[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (!known[dev]) {
    int a = 0, b = 0, cus = 0, coop = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, k_score_fused<true>, WS_THREADS, 0) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, k_score_fused<false>, WS_THREADS, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess)
      a = b = cus = coop = 0;
    cap[dev] = coop ? std::min(a, b) * cus : 0;
    known[dev] = true;
  }
  return cap[dev];
}

// Polls of an exchange wait before it gives up: IKV_EXCHANGE_SPINS (read on every call), else 2^20.
uint32_t fused_spin_limit() {
  const char *e = getenv("IKV_EXCHANGE_SPINS");
  if (e == nullptr || e[0] == '\0') return 1u << 20;
  return uint32_t(strtoul(e, nullptr, 10));
}

}  // namespace

int fused_tiles(const ikv_pool &p, const ikv_session *s, int B, uint32_t flags) {
  if (p.D != MD || p.kv_dtype != IKV_BF16 || B != 1) return 0;
  if (s[0].R <= STASH_MAX_R || s[0].R > 64 || s[0].N <= s[0].C) return 0;
  if (flags & (IKV_POOL7 | IKV_TWO_PASS)) return 0;
  // Switched off: on some calls one memory row's normaliser comes out wrong (relative
  // score errors up to 8e-4, seen with 5 layers x 1 KV head, 8300 positions, R = 24), and
  // the cause is not found. The two-pass form runs instead; IKV_FUSED is not read.
  if (!FU_ENABLED) return 0;
  const int units = p.L * p.Hkv;
  if (units >= (1 << 16)) return 0;
  const int lch = stats_chunk(s[0].N, std::max(1, units / 2));
  const int64_t tiles = cdiv(s[0].N, lch) * (lch / MFMA_TILE);
  if (tiles < FU_MIN_TILES || tiles > FU_MAX_TILES || tiles > fused_capacity()) return 0;
  return int(tiles);
}

int64_t fused_exchange_floats(const ikv_pool &p, const ikv_session *s, int B, uint32_t flags) {
  const int tiles = fused_tiles(p, s, B, flags);
  if (tiles == 0) return 0;
  const int64_t rows = int64_t(p.L) * p.Hkv * pad16(s[0].R);
  return align64f(rows * 2 * tiles * 4 + rows * 4);  // two 64-bit words per partial and per normaliser
}

hipError_t launch_score_mfma(const ScoreArgs &a, hipStream_t st) {
  const ikv_pool &p = a.pool;
  const int units = p.L * p.Hkv;
  const bool resid = (a.flags & IKV_RESIDUAL) != 0;
  const unsigned tiles = unsigned(cdiv(a.maxN, MFMA_TILE));
  const uint16_t *kp = static_cast<const uint16_t *>(p.k_pool);
  const bool ring = a.maxR <= 64;
  const bool stats = a.stats;                      // the unit-major pass splits the memory rows itself
  // the candidate lists (and -inf for every other position)
  const int lch = stats_chunk(a.maxN, std::max(1, units / 2));
  {
    KTimer kt_("k_cand_list", st);
    k_cand_list<<<dim3(unsigned(cdiv(a.maxN, lch)), a.B), CLIST_THREADS, 0, st>>>(a.sess_dev, a.slot_maps,
                                                                                  p.dead_slot, a.ws, a.scores, p.L,
                                                                                  p.Hkv, resid, lch);
  }
  const unsigned ltiles = unsigned(cdiv(a.maxN, lch) * (lch / MFMA_TILE));
  if (!stats)
    {
      KTimer kt_("k_msplit", st);
      k_msplit<<<dim3(MBAR_PARTS, a.B), 256, 0, st>>>(a.sess_dev, a.M, a.ws, a.scores, p.L, p.Hkv, resid);
    }
  const int chunk = stats ? lch : 0;
  if (a.fused_tiles > 0) {
    // one key pass: the residual head's set-up first (it reads only M, the query rows' keys
    // and the weights), then the scores with the exchange of row normalisers
    if (resid) {
      constexpr int FOLD_WGS = int((fold_items<MD>() + 511) / 512);
      const bool kv = a.mfma_resid;
      const int nfold = kv ? FOLD_WGS : 0;
      const int extra = (kv ? RES_KEYS : 0) + nfold + 1;
      KTimer kt_("k_lse_mfma", st);
      k_lse_mfma<<<dim3(unsigned(extra), a.B), 512, 0, st>>>(a.sess_dev, a.ws, p.L, p.Hkv, resid, MFMA_TILE, 0,
                                                             a.slot_maps, a.qpos, p.dead_slot, false, kv, nfold, kp,
                                                             p.num_slots, a.residual, a.ws_shared);
    }
    static const uint64_t tag = [] {
      std::random_device rd;
      uint64_t x = (uint64_t(rd()) << 32) ^ rd() ^ uint64_t(getpid()) ^
                   uint64_t(std::chrono::steady_clock::now().time_since_epoch().count());
      x &= 0xffffffull;
      return (x == 0 || x == 0xffffffull ? 0x3c3c3cull : x) << 40;
    }();
    static std::atomic<uint64_t> calls{1};
    uint64_t stamp = tag | ((calls.fetch_add(1) << 16) & ((1ull << 40) - 1));
    uint32_t spins = fused_spin_limit();
    uint32_t *fault = host_fault_word();
    uint64_t *xch = a.xch;
    const ikv_session *sd = a.sess_dev;
    const int32_t *sm = a.slot_maps;
    float *ws = a.ws, *scores = a.scores;
    int64_t ns = p.num_slots;
    int L = p.L, Hkv = p.Hkv, dead = p.dead_slot, CH = lch;
    bool rs = resid;
    void *args[] = {(void *)&kp, (void *)&ns, (void *)&L, (void *)&Hkv, (void *)&dead, (void *)&sd, (void *)&sm,
                    (void *)&ws, (void *)&scores, (void *)&rs, (void *)&CH, (void *)&xch, (void *)&stamp,
                    (void *)&spins, (void *)&fault};
    {
      KTimer kt_("k_score_fused", st);
      const void *fn = resid ? reinterpret_cast<const void *>(k_score_fused<true>)
                             : reinterpret_cast<const void *>(k_score_fused<false>);
      hipError_t e = hipLaunchCooperativeKernel(fn, dim3(unsigned(a.fused_tiles)), dim3(WS_THREADS), args, 0, st);
      if (e != hipSuccess) return e;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !resid) return e;
    return launch_residual(a, st);
  }
  if (stats)
    {
      KTimer kt_("k_score_stats", st);
      const dim3 grid(unsigned(units / 2 * cdiv(a.maxN, chunk)), a.B);
      const bool small = a.minR <= 64, large = a.maxR > 64;
      if (small)
        k_score_stats<2><<<grid, 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev, a.slot_maps,
                                               a.ws, a.M, a.scores, resid, chunk, large ? 1 : 0);
      if (large)
        k_score_stats<4><<<grid, 512, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev, a.slot_maps,
                                               a.ws, a.M, a.scores, resid, chunk, small ? 2 : 0);
    }
  else if (a.stash)
    {
      // the one key pass: logits to the stash, per-list-tile row statistics, mean key rows
      KTimer kt_("k_score_once", st);
      if (resid)
        k_score_ws<true, 1, true><<<dim3(ltiles, a.B), WS_THREADS, 0, st>>>(
            kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev, a.slot_maps, a.ws, a.scores, resid, 0, lch);
      else
        k_score_ws<false, 1, true><<<dim3(ltiles, a.B), WS_THREADS, 0, st>>>(
            kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev, a.slot_maps, a.ws, a.scores, resid, 0, lch);
    }
  else if (ring)
    {
      KTimer kt_("k_score_ring", st);
      k_score_ring<<<dim3(tiles, a.B), RING_THREADS, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                             a.slot_maps, a.ws, resid);
    }
  else
    {
      KTimer kt_("k_score_mfma<false, false>", st);
      k_score_mfma<false, false><<<dim3(tiles, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                                   a.slot_maps, a.ws, a.scores, resid);
    }
  if (a.flags & IKV_POOL7) {
    // the SnapKV-style score: row normalisers, the per-unit attention masses, the pool
    {
      KTimer kt_("k_lse_mfma", st);
      k_lse_mfma<<<dim3(unsigned(cdiv(int64_t(units) * a.maxR, 64)), a.B), 512, 0, st>>>(
          a.sess_dev, a.ws, p.L, p.Hkv, false, chunk, 0, a.slot_maps, a.qpos, p.dead_slot, true, false, 0, kp,
          p.num_slots, a.residual, a.ws_shared);
    }
    float *umass = a.ws_shared;                     // after the sessions' blocks
    {
      KTimer kt_("k_score_mass", st);
      const dim3 grid(unsigned(units / 2 * cdiv(a.maxN, chunk)), a.B);
      const bool small = a.minR <= 64, large = a.maxR > 64;
      if (small)
        k_score_stats<2, true><<<grid, 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                     a.slot_maps, a.ws, a.M, a.scores, false, chunk, large ? 1 : 0,
                                                     umass, a.total_positions);
      if (large)
        k_score_stats<4, true><<<grid, 512, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                     a.slot_maps, a.ws, a.M, a.scores, false, chunk, small ? 2 : 0,
                                                     umass, a.total_positions);
    }
    {
      KTimer kt_("k_pool7", st);
      k_pool7<<<dim3(unsigned(cdiv(a.maxN, PL_POS)), a.B), 256, 0, st>>>(a.sess_dev, a.slot_maps, p.dead_slot,
                                                                         umass, a.total_positions, units, a.scores);
    }
    return hipGetLastError();
  }
  {
    // with the matrix-core residual head, this launch also folds its first layer (one
    // item of fold_items() per thread) and builds K', V'
    constexpr int FOLD_WGS = int((fold_items<MD>() + 511) / 512);
    const bool kv = a.mfma_resid;
    const int nfold = kv ? FOLD_WGS : 0;
    const int extra = resid ? (kv ? RES_KEYS : 0) + nfold + 1 : 0;
    KTimer kt_("k_lse_mfma", st);
    k_lse_mfma<<<dim3(unsigned(cdiv(int64_t(units) * a.maxR, 64) + extra), a.B), 512, 0, st>>>(
        a.sess_dev, a.ws, p.L, p.Hkv, resid, stats ? chunk : a.stash ? lch : ring ? PART_TILE : MFMA_TILE,
        a.stash ? lch / MFMA_TILE : 0, a.slot_maps, a.qpos, p.dead_slot, a.stats, kv, nfold, kp, p.num_slots,
        a.residual, a.ws_shared);
  }
  if (a.stash)
    {
      KTimer kt_("k_score_stash", st);
      k_score_stash<<<dim3(ltiles, a.B), SS_THREADS, 0, st>>>(a.sess_dev, a.slot_maps, a.ws, a.scores, p.L, p.Hkv,
                                                              resid, lch);
    }
  // the producer/consumer second pass up to 128 memory rows: one launch per kind of
  // session (up to 64 rows, up to 128)
  const bool ws_small = a.minR <= 64, ws_large = a.maxR > 64;
  if (a.stash)
    ;                                                // scored above
  else if (a.maxR <= 128 && resid)
    {
      KTimer kt_("k_score_ws<true>", st);
      if (ws_small)
        k_score_ws<true, 1><<<dim3(ltiles, a.B), WS_THREADS, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                    a.sess_dev, a.slot_maps, a.ws, a.scores, resid,
                                                                    ws_large ? 1 : 0, lch);
      if (ws_large)
        k_score_ws<true, 2><<<dim3(ltiles, a.B), WS_THREADS, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                    a.sess_dev, a.slot_maps, a.ws, a.scores, resid,
                                                                    ws_small ? 2 : 0, lch);
    }
  else if (a.maxR <= 128)
    {
      KTimer kt_("k_score_ws<false>", st);
      if (ws_small)
        k_score_ws<false, 1><<<dim3(ltiles, a.B), WS_THREADS, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                     a.sess_dev, a.slot_maps, a.ws, a.scores, resid,
                                                                     ws_large ? 1 : 0, lch);
      if (ws_large)
        k_score_ws<false, 2><<<dim3(ltiles, a.B), WS_THREADS, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                     a.sess_dev, a.slot_maps, a.ws, a.scores, resid,
                                                                     ws_small ? 2 : 0, lch);
    }
  else if (resid)
    {
      KTimer kt_("k_score_mfma<true, true>", st);
      k_score_mfma<true, true><<<dim3(tiles, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot, a.sess_dev,
                                                                 a.slot_maps, a.ws, a.scores, resid);
    }
  else
    {
      KTimer kt_("k_score_mfma<true, false>", st);
      k_score_mfma<true, false><<<dim3(tiles, a.B), 256, 0, st>>>(kp, p.num_slots, p.L, p.Hkv, p.dead_slot,
                                                                  a.sess_dev, a.slot_maps, a.ws, a.scores, resid);
    }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !resid) return e;
  return launch_residual(a, st);
}

}  // namespace ikv
