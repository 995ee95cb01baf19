// The compact apply path (Sec. 3.4: the standard compactors left-pack the kept rows
// and re-index RoPE; the Appendix layout ablation, Table 7, compares it with the
// dead-slot redirect). The t-th kept position j of a session moves to position t and
// to the caller's destination slot dst[t]: on every layer and KV head its key is
// re-rotated by t - j (Neox rotate-half: channel pair (i, i + D/2) turns by
// (t - j) * base^(-2i/D)) and its value copied.
//
//   k_compact_list  one workgroup per session: the kept positions in position order
//                   (ballot prefix sums over 1024-position rounds), and their count;
//   k_compact_copy  one workgroup per kept index: the pair angles in float64 (they
//                   reach 1e5 radians at long distances), cos / sin in LDS, then every
//                   layer's key rows rotated in float32 and rounded once to the pool's
//                   type, value rows copied.
#include <math.h>

#include "ikv_internal.hpp"

namespace ikv {

constexpr int CL_THREADS = 1024;

__global__ void __launch_bounds__(CL_THREADS) k_compact_list(const ikv_session *__restrict__ sess,
                                                             const int32_t *__restrict__ slot_maps, int dead,
                                                             const uint8_t *__restrict__ keep,
                                                             int32_t *__restrict__ pos_list,
                                                             int32_t *__restrict__ n_keep) {
  __shared__ int wsum[CL_THREADS / WAVE];
  __shared__ int base_s;
  const int b = blockIdx.x;
  const ikv_session s = sess[b];
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  if (t == 0) base_s = 0;
  __syncthreads();
  for (int j0 = 0; j0 < s.N; j0 += CL_THREADS) {
    const int j = j0 + t;
    const bool k = j < s.N && keep[s.slot_off + j] && slot_maps[s.slot_off + j] != dead;
    const uint64_t m = __ballot(k);
    const int below = __popcll(m & ((uint64_t(1) << lane) - 1));
    if (lane == 0) wsum[w] = __popcll(m);
    __syncthreads();
    int off = base_s;
    for (int q = 0; q < w; ++q) off += wsum[q];
    if (k) pos_list[s.slot_off + off + below] = j;
    __syncthreads();
    if (t == 0) {
      int tot = 0;
      for (int q = 0; q < CL_THREADS / WAVE; ++q) tot += wsum[q];
      base_s += tot;
    }
    __syncthreads();
  }
  if (t == 0) n_keep[b] = base_s;
}

constexpr int CC_THREADS = 256;
constexpr int CC_PP = 4;                         // channel pairs per thread per step

// four consecutive channels: one 8-byte access (bf16) or one 16-byte access (float32);
// stores round to the pool's type (nearest even for bf16)
__device__ __forceinline__ void ld4(const uint16_t *p, float *x) {
  const uint2 v = *reinterpret_cast<const uint2 *>(p);
  x[0] = __uint_as_float(v.x << 16);
  x[1] = __uint_as_float(v.x & 0xffff0000u);
  x[2] = __uint_as_float(v.y << 16);
  x[3] = __uint_as_float(v.y & 0xffff0000u);
}
__device__ __forceinline__ void ld4(const float *p, float *x) {
  const float4 v = *reinterpret_cast<const float4 *>(p);
  x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
}
__device__ __forceinline__ void st4(uint16_t *p, const float *y) {
  *reinterpret_cast<uint2 *>(p) =
      make_uint2(uint32_t(float_to_bf16_bits(y[0])) | (uint32_t(float_to_bf16_bits(y[1])) << 16),
                 uint32_t(float_to_bf16_bits(y[2])) | (uint32_t(float_to_bf16_bits(y[3])) << 16));
}
__device__ __forceinline__ void st4(float *p, const float *y) {
  *reinterpret_cast<float4 *>(p) = make_float4(y[0], y[1], y[2], y[3]);
}
__device__ __forceinline__ void cp4(uint16_t *d, const uint16_t *s) {
  *reinterpret_cast<uint2 *>(d) = *reinterpret_cast<const uint2 *>(s);
}
__device__ __forceinline__ void cp4(float *d, const float *s) {
  *reinterpret_cast<float4 *>(d) = *reinterpret_cast<const float4 *>(s);
}

template <typename T>
__global__ void __launch_bounds__(CC_THREADS) k_compact_copy(const ikv_session *__restrict__ sess, T *__restrict__ kp,
                                                             T *__restrict__ vp, int64_t num_slots, int L, int Hkv,
                                                             int D, const int32_t *__restrict__ slot_maps,
                                                             const int32_t *__restrict__ dst,
                                                             const int32_t *__restrict__ pos_list,
                                                             const int32_t *__restrict__ n_keep, double base) {
  __shared__ float cs[64], sn[64];
  const int b = blockIdx.y;
  const ikv_session s = sess[b];
  const int tk = blockIdx.x;
  if (tk >= n_keep[b]) return;
  const int j = pos_list[s.slot_off + tk];
  const int64_t src = slot_maps[s.slot_off + j], dslot = dst[s.slot_off + tk];
  const int h = D / 2, t = threadIdx.x;
  if (t < h) {
    const double ang = double(tk - j) * pow(base, -2.0 * double(t) / double(D));
    cs[t] = float(cos(ang));
    sn[t] = float(sin(ang));
  }
  __syncthreads();
  const int64_t row = int64_t(Hkv) * D;          // elements of one slot in one layer
  const int groups = Hkv * (h / CC_PP);          // pair groups per layer
  for (int g = t; g < L * groups; g += CC_THREADS) {
    const int l = g / groups, r = g - l * groups;
    const int hd = r / (h / CC_PP), q = (r - hd * (h / CC_PP)) * CC_PP;
    const int64_t o_src = (int64_t(l) * num_slots + src) * row + int64_t(hd) * D;
    const int64_t o_dst = (int64_t(l) * num_slots + dslot) * row + int64_t(hd) * D;
    float x1[CC_PP], x2[CC_PP], y1[CC_PP], y2[CC_PP];
    ld4(kp + o_src + q, x1);
    ld4(kp + o_src + h + q, x2);
#pragma unroll
    for (int e = 0; e < CC_PP; ++e) {
      const float c = cs[q + e], sv = sn[q + e];
      y1[e] = x1[e] * c - x2[e] * sv;
      y2[e] = x2[e] * c + x1[e] * sv;
    }
    st4(kp + o_dst + q, y1);
    st4(kp + o_dst + h + q, y2);
    cp4(vp + o_dst + q, vp + o_src + q);
    cp4(vp + o_dst + h + q, vp + o_src + h + q);
  }
}

hipError_t launch_compact(const ikv_pool &pool, const ikv_session *sess_dev, int B, int maxN,
                          const int32_t *slot_maps, const uint8_t *keep, const int32_t *dst, double base,
                          int32_t *n_keep, int32_t *pos_list, hipStream_t st) {
  {
    KTimer kt_("k_compact_list", st);
    k_compact_list<<<B, CL_THREADS, 0, st>>>(sess_dev, slot_maps, pool.dead_slot, keep, pos_list, n_keep);
  }
  if (maxN > 0) {
    KTimer kt_("k_compact_copy", st);
    const dim3 grid(unsigned(maxN), B);
    if (pool.kv_dtype == IKV_BF16)
      k_compact_copy<uint16_t><<<grid, CC_THREADS, 0, st>>>(
          sess_dev, static_cast<uint16_t *>(pool.k_pool), static_cast<uint16_t *>(pool.v_pool), pool.num_slots, pool.L,
          pool.Hkv, pool.D, slot_maps, dst, pos_list, n_keep, base);
    else
      k_compact_copy<float><<<grid, CC_THREADS, 0, st>>>(
          sess_dev, static_cast<float *>(pool.k_pool), static_cast<float *>(pool.v_pool), pool.num_slots, pool.L,
          pool.Hkv, pool.D, slot_maps, dst, pos_list, n_keep, base);
  }
  return hipGetLastError();
}

}  // namespace ikv
