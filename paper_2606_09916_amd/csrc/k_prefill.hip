// Prefill of the actionable query span (Sec. 3.5: the post-RoPE Q and K the retention
// step needs are the ones the model's own attention computes; Sec. 3.2: Enc(q_t) is
// the mean of the span's post-RoPE Q rows; Eq. 6: the cross-attention keys are the
// mean key rows at the query positions). One call per turn, before the retention step:
//
//   k_prefill_rope  one workgroup per (layer, span token, session): Neox RoPE at the
//                   token's position (pair angles in float64, cos / sin in LDS, rotation
//                   in float32, one rounding to the pool's type) of the query rows
//                   (written out) and key rows (written into the pool at the token's
//                   slot, with the value rows); the sum of its rotated key rows over the
//                   KV heads (this layer's part of the mean key row);
//   k_prefill_memory with a memory, Eq. 2 per (layer, head): Enc from the rotated query
//                   rows as written, summed in token order;
//   k_prefill_attn  one workgroup per (layer, KV head, session, split of the keys):
//                   causal attention of the span's query rows of the KV head's G query
//                   heads over the history slots and the span's own slots (matrix
//                   cores, below); k_prefill_merge combines the splits;
//   k_prefill_kq    the mean key rows of the span tokens: the layers' parts summed in
//                   layer order.
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int PD = 128;                          // head dimension of the attention kernel
constexpr int PR_THREADS = 256;
constexpr int PR_KMAX = 2048;                    // Hkv * D: key channels of a layer

// Per session b: n = qe - qs span tokens; the packed inputs and outputs of the sessions
// before b: rows of q (Hq per layer) and of k / v (Hkv per layer), and the mean key rows.
__device__ __forceinline__ void prefill_offsets(const ikv_session *sess, int b, int L, int Hq, int Hkv, int D,
                                                int64_t *q_off, int64_t *kv_off, int64_t *kq_off) {
  int64_t nq = 0;
  for (int i = 0; i < b; ++i) nq += sess[i].qe - sess[i].qs;
  *q_off = nq * L * Hq * D;
  *kv_off = nq * L * Hkv * D;
  *kq_off = nq * D;
}

// One workgroup per (layer, span token, session): the token's angles, its rotated query
// rows (written out), its rotated key rows (into the pool at the token's slot, with the
// value rows) and this layer's part of its mean key row (the rotated key rows summed
// over the KV heads in order).
template <typename T>
__global__ void __launch_bounds__(PR_THREADS) k_prefill_rope(const ikv_session *__restrict__ sess, int L, int Hq,
                                                             int Hkv, int D, T *__restrict__ kpool,
                                                             T *__restrict__ vpool, int64_t num_slots,
                                                             const int32_t *__restrict__ slot_maps,
                                                             const T *__restrict__ q_raw, const T *__restrict__ k_raw,
                                                             const T *__restrict__ v_raw, T *__restrict__ q_out,
                                                             double base, float *__restrict__ kq_part) {
  __shared__ float cs[64], sn[64];
  __shared__ float ksum[PR_KMAX];                // this token's rotated key rows [Hkv][D]
  const int l = blockIdx.x, t = blockIdx.y, b = blockIdx.z;
  const ikv_session s = sess[b];
  const int n = s.qe - s.qs;
  if (t >= n) return;
  int64_t q_off, kv_off, kq_off;
  prefill_offsets(sess, b, L, Hq, Hkv, D, &q_off, &kv_off, &kq_off);
  const int t0 = threadIdx.x, h2 = D / 2;
  const int pos = s.qs + t;
  if (t0 < h2) {
    const double ang = double(pos) * pow(base, -2.0 * double(t0) / double(D));
    cs[t0] = float(cos(ang));
    sn[t0] = float(sin(ang));
  }
  __syncthreads();
  // query rows: element e = (head, channel); channel c < D/2 pairs with c + D/2
  const int nq_el = Hq * D, nk_el = Hkv * D;
  for (int e = t0; e < nq_el; e += PR_THREADS) {
    const int h = e / D, c = e - h * D, i = c < h2 ? c : c - h2;
    const int64_t base_row = q_off + ((int64_t(l) * Hq + h) * n + t) * D;
    const float x = Store<T>::ld(q_raw + base_row + c);
    const float y = Store<T>::ld(q_raw + base_row + (c < h2 ? c + h2 : c - h2));
    const float r = c < h2 ? x * cs[i] - y * sn[i] : x * cs[i] + y * sn[i];
    q_out[base_row + c] = Store<T>::from(r);
  }
  // key rows into the pool at the token's slot, value rows copied
  const int64_t slot = slot_maps[s.slot_off + pos];
  for (int e = t0; e < nk_el; e += PR_THREADS) {
    const int h = e / D, c = e - h * D, i = c < h2 ? c : c - h2;
    const int64_t src = kv_off + ((int64_t(l) * Hkv + h) * n + t) * D;
    const float x = Store<T>::ld(k_raw + src + c);
    const float y = Store<T>::ld(k_raw + src + (c < h2 ? c + h2 : c - h2));
    const float r = c < h2 ? x * cs[i] - y * sn[i] : x * cs[i] + y * sn[i];
    const T rv = Store<T>::from(r);
    const int64_t dst = ((int64_t(l) * num_slots + slot) * Hkv + h) * D + c;
    kpool[dst] = rv;
    vpool[dst] = v_raw[src + c];
    ksum[e] = Store<T>::ld(&rv);
  }
  __syncthreads();
  // this layer's part of the token's mean key row: the rotated rows summed over KV heads in order
  for (int c = t0; c < D; c += PR_THREADS) {
    float a = 0.f;
    for (int h = 0; h < Hkv; ++h) a += ksum[h * D + c];
    kq_part[(kq_off * L) + (int64_t(l) * n + t) * D + c] = a;
  }
}

// Eq. 2 for memory row h of layer l (one per query head): Enc is the mean over the span
// of the rotated query rows as written (summed in token order), M <- decay M + Enc, then
// the row divided by max(||row||, 1e-12) (the squares summed in a fixed tree order).
// Workgroup (layer, head, session); thread c is channel c.
template <typename T>
__global__ void __launch_bounds__(PD) k_prefill_memory(const ikv_session *__restrict__ sess, int L, int Hq, int Hkv,
                                                       const T *__restrict__ q_out, float *__restrict__ M,
                                                       float decay) {
  __shared__ float red[PD];
  const int l = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const ikv_session s = sess[b];
  const int n = s.qe - s.qs;
  if (n <= 0) return;
  int64_t q_off, kv_off, kq_off;
  prefill_offsets(sess, b, L, Hq, Hkv, PD, &q_off, &kv_off, &kq_off);
  const int c = threadIdx.x;
  const T *qr = q_out + q_off + (int64_t(l) * Hq + h) * n * PD + c;
  float enc = 0.f;
  for (int t = 0; t < n; ++t) enc += Store<T>::ld(qr + int64_t(t) * PD);
  float *Mr = M + s.mem_off + (int64_t(l) * Hq + h) * PD;
  const float v = decay * Mr[c] + enc * (1.0f / float(n));
  red[c] = v * v;
  __syncthreads();
  for (int off = PD / 2; off > 0; off >>= 1) {
    if (c < off) red[c] += red[c + off];
    __syncthreads();
  }
  Mr[c] = v / fmaxf(sqrtf(red[0]), 1e-12f);
}

// ------------------------------------------------------------------ causal attention
// Workgroup (layer l, KV head g, session b, split z), eight waves: query row
// r = h' n + t (h' the query head within the group, t the span token) belongs to wave
// r / 32, as row r % 16 of its row block (r / 16) % 2; each key and value fragment a
// wave reads from LDS feeds the MFMAs of both its row blocks. The keys (the history slots, then the span's slots) are cut into 64-key
// tiles and the tiles into `nsplit` contiguous runs, one per split, so that a long
// history fills the chip. Per tile a wave computes S^T = K Q^T (16 keys x 16 rows per
// MFMA block, bf16 inputs exact, float32 accumulation), keeps an online (max, sum) per
// row, and adds O^T += V^T P^T, the weights P split into bf16 hi + lo (two MFMAs;
// 2^-17 relative). The weights of keys 16 kb + 4 g + i that a lane holds are already
// the B operand of the second product, up to the order of the contraction index
// (perm32): the transposed value tile in LDS is read in that order. Key rows stay as
// loaded (rows of 136 bf16); value rows are written transposed (rows of 72 bf16 per
// channel).
// Loads: two tiles in registers beyond the one in LDS. While tile i is computed, tile
// i + 1 is on its way and tile i + 2 is issued, and the slot ids of tile i + 3 load
// before it. Every iteration issues the same loads whatever the split's length (past
// the keys' end the first span slot is read and masked), so the compiler's memory
// waits are exact counts.
// With one split the rows are written normalised; with more, each split writes its
// unnormalised rows and (max, sum) and k_prefill_merge combines them.
constexpr int PA_WAVES = 8;
constexpr int PA_THREADS = PA_WAVES * WAVE;
constexpr int PA_TILE = 64;
constexpr int PA_KROW = PD + 8;
constexpr int PA_VROW = PA_TILE + 8;
constexpr int PA_ROWS = 256;                     // query rows of a (layer, KV head) at most: n G <= 256
constexpr int PA_RB = 2;                         // 16-row blocks per wave: 32 rows, so each key and
                                                 // value fragment read from LDS feeds two MFMAs
// The transposed value tile stores key k of channel ch at k ^ vt_swz(ch): a multiple of
// 4 that changes with the channel group, so four consecutive keys stay adjacent (one
// 8-byte read) while the 16-bit stores of a wave's 16 channel groups spread over the
// LDS banks instead of landing on four of them.
__device__ __forceinline__ int vt_swz(int ch) { return ((ch >> 3) & 15) << 2; }

template <bool PART>
__global__ void __launch_bounds__(PA_THREADS) k_prefill_attn(const ikv_session *__restrict__ sess, int L, int Hq,
                                                             int Hkv, const uint16_t *__restrict__ kpool,
                                                             const uint16_t *__restrict__ vpool, int64_t num_slots,
                                                             const int32_t *__restrict__ slot_maps,
                                                             const int32_t *__restrict__ hist,
                                                             const int32_t *__restrict__ n_hist,
                                                             const uint16_t *__restrict__ q_rot,
                                                             uint16_t *__restrict__ out, float *__restrict__ part_o,
                                                             float *__restrict__ part_ml) {
  __shared__ __align__(16) uint16_t ks[2][PA_TILE * PA_KROW];
  __shared__ __align__(16) uint16_t vt[2][PD * PA_VROW];
  const int lg = blockIdx.x, b = blockIdx.y, split = blockIdx.z, nsplit = gridDim.z;
  const int l = lg / Hkv, g_kv = lg - l * Hkv;
  const ikv_session s = sess[b];
  const int n = s.qe - s.qs;
  if (n <= 0) return;
  const int G = Hq / Hkv, nrows = n * G;
  int64_t q_off, kv_off, kq_off;
  prefill_offsets(sess, b, L, Hq, Hkv, PD, &q_off, &kv_off, &kq_off);
  const int nh = n_hist[b];
  const int T = nh + n;                           // keys: history, then the span
  const int ntile_all = (T + PA_TILE - 1) / PA_TILE;
  const int tps = (ntile_all + nsplit - 1) / nsplit;
  const int tb = min(ntile_all, split * tps), te = min(ntile_all, tb + tps);
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int g = lane >> 4, c = lane & 15;
  // this lane's query rows, one per 16-row block (clamped; the extra rows are never written)
  int hq[PA_RB], tr[PA_RB];
#pragma unroll
  for (int rb = 0; rb < PA_RB; ++rb) {
    const int row = min(32 * w + 16 * rb + c, nrows - 1);
    hq[rb] = row / n;
    tr[rb] = row - hq[rb] * n;
  }
  const bool wave_on = 32 * w < nrows;
  const float scale = 1.4426950408889634f / sqrtf(float(PD));

  float m_run[PA_RB], l_run[PA_RB];              // per row block: this lane's row (rows are the lane index c)
  f32x4 o[PA_RB][8];                              // O^T blocks: channel 16 db + 4 g + i, row c
#pragma unroll
  for (int rb = 0; rb < PA_RB; ++rb) {
    m_run[rb] = -INFINITY;
    l_run[rb] = 0.f;
#pragma unroll
    for (int db = 0; db < 8; ++db) o[rb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  if (tb < te) {
    // query fragments (B operand of S^T): row block rb, channels 32 ks + 8 g .. + 8
    bf16x8 qf[PA_RB][4];
#pragma unroll
    for (int rb = 0; rb < PA_RB; ++rb) {
      const uint16_t *qr = q_rot + q_off + ((int64_t(l) * Hq + g_kv * G + hq[rb]) * n + tr[rb]) * PD;
#pragma unroll
      for (int ks4 = 0; ks4 < 4; ++ks4) qf[rb][ks4] = *reinterpret_cast<const bf16x8 *>(qr + 32 * ks4 + 8 * g);
    }
    const int32_t *S = slot_maps + s.slot_off;
    const int32_t *H = hist + s.slot_off;
    // tile loads: thread t takes keys t / 16 and t / 16 + 32 of the tile, 16-byte chunk
    // t % 16 of their K and V rows
    const int lk = t >> 4, lc = t & 15;
    // the slots of this thread's two keys in tile `tile`: one load each from the history
    // list or the span's slots (past the keys' end, the first span slot: a valid row,
    // masked out)
    auto tile_slot = [&](int tile, int half) __attribute__((always_inline)) -> int32_t {
      const int kk = tile * PA_TILE + lk + 32 * half;
      const int32_t *p = kk < nh ? H + kk : S + s.qs + (kk < T ? kk - nh : 0);
      return *p;
    };
    const int64_t lbase = (int64_t(l) * num_slots * Hkv + g_kv) * PD + lc * 8;
    struct Regs { uint4 k0, v0, k1, v1; };     // keys lk and lk + 32 (plain members: kept in registers)
    struct Slots { int32_t s0, s1; };
    auto slots = [&](int tile) __attribute__((always_inline)) { return Slots{tile_slot(tile, 0), tile_slot(tile, 1)}; };
    auto load_kv = [&](const Slots &sl, Regs &r) __attribute__((always_inline)) {
      const int64_t o0 = lbase + int64_t(sl.s0) * Hkv * PD, o1 = lbase + int64_t(sl.s1) * Hkv * PD;
      r.k0 = *reinterpret_cast<const uint4 *>(kpool + o0);
      r.v0 = *reinterpret_cast<const uint4 *>(vpool + o0);
      r.k1 = *reinterpret_cast<const uint4 *>(kpool + o1);
      r.v1 = *reinterpret_cast<const uint4 *>(vpool + o1);
    };
    auto store_one = [&](int stg, int key, const uint4 &kr, const uint4 &vr) __attribute__((always_inline)) {
      *reinterpret_cast<uint4 *>(&ks[stg][key * PA_KROW + lc * 8]) = kr;
      const uint32_t wv[4] = {vr.x, vr.y, vr.z, vr.w};
      const int kp = key ^ vt_swz(lc * 8);          // channels lc*8 .. +7 share one swizzle
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vt[stg][(lc * 8 + 2 * e) * PA_VROW + kp] = uint16_t(wv[e] & 0xffffu);
        vt[stg][(lc * 8 + 2 * e + 1) * PA_VROW + kp] = uint16_t(wv[e] >> 16);
      }
    };
    auto store_tile = [&](int stg, const Regs &r) __attribute__((always_inline)) {
      store_one(stg, lk, r.k0, r.v0);
      store_one(stg, lk + 32, r.k1, r.v1);
    };
    auto compute = [&](int stg, int tile) __attribute__((always_inline)) {
      if (!wave_on) return;
      const bool hist_tile = (tile + 1) * PA_TILE <= nh;   // wave-uniform
      // S^T: key blocks kb (keys 16 kb .. + 15), lane (g, c): keys 16 kb + 4 g + i, row c of block rb
      f32x4 sacc[PA_RB][4];
#pragma unroll
      for (int rb = 0; rb < PA_RB; ++rb)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) sacc[rb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const uint16_t *kr = &ks[stg][(16 * kb + c) * PA_KROW];
#pragma unroll
        for (int ks4 = 0; ks4 < 4; ++ks4) {
          const bf16x8 kfr = *reinterpret_cast<const bf16x8 *>(kr + 32 * ks4 + 8 * g);
#pragma unroll
          for (int rb = 0; rb < PA_RB; ++rb)
            sacc[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kfr, qf[rb][ks4], sacc[rb][kb], 0, 0, 0);
        }
      }
      // per row block: mask (keys past the end; span keys after the row's token), the
      // online softmax, and the weights split into bf16 hi + lo for the second product
      bf16x8 ph[PA_RB][2], pl[PA_RB][2];
#pragma unroll
      for (int rb = 0; rb < PA_RB; ++rb) {
        float tmax = -INFINITY;
        if (hist_tile) {                            // every key of the tile is history: nothing masked,
#pragma unroll                                      // the maximum taken on the raw logits
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) tmax = fmaxf(tmax, sacc[rb][kb][i]);
        } else {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int kk = tile * PA_TILE + 16 * kb + 4 * g + i;
              const bool ok = kk < T && (kk < nh || kk - nh <= tr[rb]);
              const float x = ok ? sacc[rb][kb][i] * scale : -INFINITY;
              sacc[rb][kb][i] = x;
              tmax = fmaxf(tmax, x);
            }
        }
        tmax = fmaxf(tmax, __shfl_xor(tmax, 16, WAVE));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, WAVE));
        if (hist_tile) tmax *= scale;               // scale > 0: the same value as the maximum of the scaled logits
        const float m_new = fmaxf(m_run[rb], tmax);
        // a row with no key yet (m_new = -inf) keeps zero weights and sums
        const float corr = m_run[rb] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[rb] - m_new);
        float psum = 0.f;
        float p[4][4];
        if (hist_tile) {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              p[kb][i] = __builtin_amdgcn_exp2f(fmaf(sacc[rb][kb][i], scale, -m_new));
              psum += p[kb][i];
            }
        } else {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              p[kb][i] = sacc[rb][kb][i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sacc[rb][kb][i] - m_new);
              psum += p[kb][i];
            }
        }
        psum += __shfl_xor(psum, 16, WAVE);
        psum += __shfl_xor(psum, 32, WAVE);
        l_run[rb] = l_run[rb] * corr + psum;
        // the outputs are rescaled only when some row's maximum moved (corr = 1 otherwise)
        if (__builtin_amdgcn_ballot_w64(m_new != m_run[rb]) != 0)
#pragma unroll
          for (int db = 0; db < 8; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) o[rb][db][i] *= corr;
        m_run[rb] = m_new;
        // k index 8 g + e of 32-key step st2 stands for key perm32(g, e)
#pragma unroll
        for (int st2 = 0; st2 < 2; ++st2)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float v = e < 4 ? p[2 * st2][e] : p[2 * st2 + 1][e - 4];
            ph[rb][st2][e] = __bf16(v);
            pl[rb][st2][e] = __bf16(v - float(ph[rb][st2][e]));
          }
      }
      // O^T += V^T P^T over two 32-key steps, each value fragment shared by the row blocks
#pragma unroll
      for (int st2 = 0; st2 < 2; ++st2) {
#pragma unroll
        for (int db = 0; db < 8; ++db) {
          const uint16_t *vr = &vt[stg][(16 * db + c) * PA_VROW];
          const int sw = vt_swz(16 * db + c);
          const uint2 a = *reinterpret_cast<const uint2 *>(vr + ((32 * st2 + 4 * g) ^ sw));
          const uint2 bq = *reinterpret_cast<const uint2 *>(vr + ((32 * st2 + 16 + 4 * g) ^ sw));
          const uint4 av = make_uint4(a.x, a.y, bq.x, bq.y);
          const bf16x8 va = __builtin_bit_cast(bf16x8, av);
#pragma unroll
          for (int rb = 0; rb < PA_RB; ++rb) {
            o[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, ph[rb][st2], o[rb][db], 0, 0, 0);
            o[rb][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pl[rb][st2], o[rb][db], 0, 0, 0);
          }
        }
      }
    };
    // the same order of loads as at the top of every later pair (tile + 2's slots, then
    // tile + 1's rows), so that the waits the compiler places inside the loop stay exact
    Regs rA, rB;
    load_kv(slots(tb), rA);
    const Slots sl1 = slots(tb + 1);
    Slots sl2 = slots(tb + 2);
    __builtin_amdgcn_sched_barrier(0);
    load_kv(sl1, rB);
    __builtin_amdgcn_sched_barrier(0);
    store_tile(0, rA);
    __syncthreads();
    int tile = tb;
    for (; tile + 1 < te; tile += 2) {
      // LDS stage 0 holds `tile`; rB tile + 1; rA takes tile + 2
      const Slots sl3 = slots(tile + 3);
      __builtin_amdgcn_sched_barrier(0);
      load_kv(sl2, rA);
      __builtin_amdgcn_sched_barrier(0);
      compute(0, tile);
      store_tile(1, rB);
      __syncthreads();
      // LDS stage 1 holds tile + 1; rA tile + 2; rB takes tile + 3
      sl2 = slots(tile + 4);
      __builtin_amdgcn_sched_barrier(0);
      load_kv(sl3, rB);
      __builtin_amdgcn_sched_barrier(0);
      compute(1, tile + 1);
      store_tile(0, rA);
      __syncthreads();
    }
    if (tile < te) compute(0, tile);              // an odd last tile (its successors' loads go unused)
  }
  if (!wave_on) return;
#pragma unroll
  for (int rb = 0; rb < PA_RB; ++rb) {
    const int r = 32 * w + 16 * rb + c;
    if (r >= nrows) continue;
    if constexpr (PART) {
      // this split's rows, unnormalised, and their (max, sum); read once, by the merge:
      // non-temporal
      const int64_t pr = ((int64_t(b) * gridDim.x + lg) * nsplit + split) * PA_ROWS + r;
#pragma unroll
      for (int db = 0; db < 8; ++db)
        __builtin_nontemporal_store(o[rb][db], reinterpret_cast<f32x4 *>(part_o + pr * PD + 16 * db + 4 * g));
      if (g == 0) *reinterpret_cast<float2 *>(part_ml + pr * 2) = make_float2(m_run[rb], l_run[rb]);
    } else {
      // out[l][g_kv G + h'][t][:] = O / l
      const float inv = 1.0f / l_run[rb];
#pragma unroll
      for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          out[q_off + ((int64_t(l) * Hq + g_kv * G + hq[rb]) * n + tr[rb]) * PD + 16 * db + 4 * g + i] =
              float_to_bf16_bits(o[rb][db][i] * inv);
    }
  }
}

// The splits of each query row of the attention: with M the largest split maximum,
// out = sum_z o_z 2^(m_z - M) / sum_z l_z 2^(m_z - M) (a split that saw no key of the
// row has m = -inf and weighs zero). Workgroup (layer and KV head, session, 2 rows);
// thread (row, channel d) has every split's value and (max, sum) in flight at once.
constexpr int PM_ROWS = 2;
template <int SMAX>                              // SMAX >= nsplit: loads past nsplit re-read split 0
__global__ void __launch_bounds__(PM_ROWS * PD) k_prefill_merge(const ikv_session *__restrict__ sess, int L, int Hq,
                                                                int Hkv, int nsplit, const float *__restrict__ part_o,
                                                                const float *__restrict__ part_ml,
                                                                uint16_t *__restrict__ out) {
  const int lg = blockIdx.x, b = blockIdx.y;
  const int l = lg / Hkv, g_kv = lg - l * Hkv;
  const ikv_session s = sess[b];
  const int n = s.qe - s.qs;
  const int G = Hq / Hkv, nrows = n * G;
  const int r = blockIdx.z * PM_ROWS + threadIdx.x / PD, d = threadIdx.x % PD;
  if (r >= nrows) return;
  int64_t q_off, kv_off, kq_off;
  prefill_offsets(sess, b, L, Hq, Hkv, PD, &q_off, &kv_off, &kq_off);
  const int64_t p0 = (int64_t(b) * gridDim.x + lg) * nsplit * PA_ROWS + r;
  float oz[SMAX];
  float2 mz[SMAX];
#pragma unroll
  for (int z = 0; z < SMAX; ++z) {
    const int64_t pz = p0 + int64_t(z < nsplit ? z : 0) * PA_ROWS;
    oz[z] = __builtin_nontemporal_load(part_o + pz * PD + d);
    mz[z] = reinterpret_cast<const float2 *>(part_ml)[pz];
  }
  float M = -INFINITY;
#pragma unroll
  for (int z = 0; z < SMAX; ++z)
    if (z < nsplit) M = fmaxf(M, mz[z].x);
  float acc = 0.f, lsum = 0.f;
#pragma unroll
  for (int z = 0; z < SMAX; ++z)
    if (z < nsplit && mz[z].x != -INFINITY) {
      const float f = __builtin_amdgcn_exp2f(mz[z].x - M);
      acc = fmaf(oz[z], f, acc);
      lsum = fmaf(mz[z].y, f, lsum);
    }
  const int hq = r / n, tr = r - hq * n;
  out[q_off + ((int64_t(l) * Hq + g_kv * G + hq) * n + tr) * PD + d] = float_to_bf16_bits(acc / lsum);
}

__global__ void __launch_bounds__(128) k_prefill_kq(const ikv_session *__restrict__ sess, int L, int Hq, int Hkv,
                                                    int D, const float *__restrict__ kq_part, float *__restrict__ kq) {
  const int t = blockIdx.x, b = blockIdx.y;
  const ikv_session s = sess[b];
  const int n = s.qe - s.qs;
  if (t >= n || int(threadIdx.x) >= D) return;
  int64_t q_off, kv_off, kq_off;
  prefill_offsets(sess, b, L, Hq, Hkv, D, &q_off, &kv_off, &kq_off);
  float a = 0.f;
  for (int l = 0; l < L; ++l) a += kq_part[kq_off * L + (int64_t(l) * n + t) * D + threadIdx.x];
  kq[kq_off + int64_t(t) * D + threadIdx.x] = a / float(L * Hkv);
}

hipError_t launch_prefill(const ikv_pool &pool, const ikv_session *sess_dev, int B, int max_n, int splits,
                          const int32_t *slot_maps, const void *q_raw, const void *k_raw, const void *v_raw,
                          const int32_t *hist, const int32_t *n_hist, double base, float decay, float *M,
                          void *q_out, void *out, float *kq, float *ws, int64_t kq_floats, hipStream_t st) {
  {
    KTimer kt_("k_prefill_rope", st);
    const dim3 g1(unsigned(pool.L), unsigned(max_n), B);
    if (pool.kv_dtype == IKV_BF16)
      k_prefill_rope<uint16_t><<<g1, PR_THREADS, 0, st>>>(
          sess_dev, pool.L, pool.Hq, pool.Hkv, pool.D, static_cast<uint16_t *>(pool.k_pool),
          static_cast<uint16_t *>(pool.v_pool), pool.num_slots, slot_maps, static_cast<const uint16_t *>(q_raw),
          static_cast<const uint16_t *>(k_raw), static_cast<const uint16_t *>(v_raw), static_cast<uint16_t *>(q_out),
          base, ws);
    else
      k_prefill_rope<float><<<g1, PR_THREADS, 0, st>>>(
          sess_dev, pool.L, pool.Hq, pool.Hkv, pool.D, static_cast<float *>(pool.k_pool),
          static_cast<float *>(pool.v_pool), pool.num_slots, slot_maps, static_cast<const float *>(q_raw),
          static_cast<const float *>(k_raw), static_cast<const float *>(v_raw), static_cast<float *>(q_out), base, ws);
  }
  if (M) {
    KTimer kt_("k_prefill_memory", st);
    const dim3 gm(unsigned(pool.L), unsigned(pool.Hq), B);
    if (pool.kv_dtype == IKV_BF16)
      k_prefill_memory<uint16_t><<<gm, PD, 0, st>>>(sess_dev, pool.L, pool.Hq, pool.Hkv,
                                                     static_cast<const uint16_t *>(q_out), M, decay);
    else
      k_prefill_memory<float><<<gm, PD, 0, st>>>(sess_dev, pool.L, pool.Hq, pool.Hkv,
                                                  static_cast<const float *>(q_out), M, decay);
  }
  {
    KTimer kt_("k_prefill_attn", st);
    const dim3 grid(unsigned(pool.L * pool.Hkv), B, unsigned(splits));
    float *part_o = ws + kq_floats;
    float *part_ml = part_o + int64_t(B) * pool.L * pool.Hkv * splits * PA_ROWS * PD;
    if (splits > 1)
      k_prefill_attn<true><<<grid, PA_THREADS, 0, st>>>(
          sess_dev, pool.L, pool.Hq, pool.Hkv, static_cast<const uint16_t *>(pool.k_pool),
          static_cast<const uint16_t *>(pool.v_pool), pool.num_slots, slot_maps, hist, n_hist,
          static_cast<const uint16_t *>(q_out), static_cast<uint16_t *>(out), part_o, part_ml);
    else
      k_prefill_attn<false><<<grid, PA_THREADS, 0, st>>>(
          sess_dev, pool.L, pool.Hq, pool.Hkv, static_cast<const uint16_t *>(pool.k_pool),
          static_cast<const uint16_t *>(pool.v_pool), pool.num_slots, slot_maps, hist, n_hist,
          static_cast<const uint16_t *>(q_out), static_cast<uint16_t *>(out), nullptr, nullptr);
    if (splits > 1) {
      KTimer kt2_("k_prefill_merge", st);
      const dim3 gm(unsigned(pool.L * pool.Hkv), B, unsigned(PA_ROWS / PM_ROWS));
      uint16_t *o16 = static_cast<uint16_t *>(out);
      if (splits <= 4)
        k_prefill_merge<4><<<gm, PM_ROWS * PD, 0, st>>>(sess_dev, pool.L, pool.Hq, pool.Hkv, splits, part_o, part_ml, o16);
      else if (splits <= 8)
        k_prefill_merge<8><<<gm, PM_ROWS * PD, 0, st>>>(sess_dev, pool.L, pool.Hq, pool.Hkv, splits, part_o, part_ml, o16);
      else
        k_prefill_merge<16><<<gm, PM_ROWS * PD, 0, st>>>(sess_dev, pool.L, pool.Hq, pool.Hkv, splits, part_o, part_ml,
                                                         o16);
    }
  }
  {
    KTimer kt_("k_prefill_kq", st);
    k_prefill_kq<<<dim3(unsigned(max_n), B), 128, 0, st>>>(sess_dev, pool.L, pool.Hq, pool.Hkv, pool.D, ws, kq);
  }
  return hipGetLastError();
}

}  // namespace ikv
