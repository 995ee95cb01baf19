// Sentinel dead slot (Sec. 3.4) and the QueryMemory recurrence (Eq. 2, Sec. 3.2).
#include "ikv_internal.hpp"

namespace ikv {

// K[l][dead][h][:] = -1e4, V[l][dead][h][:] = 0 on every layer and head.
template <typename T>
__global__ void k_init_dead_slot(T *__restrict__ k, T *__restrict__ v, int L, int64_t num_slots, int HD,
                                 int dead) {
  int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= int64_t(L) * HD) return;
  int64_t l = i / HD, e = i % HD;
  int64_t off = (l * num_slots + dead) * HD + e;
  k[off] = Store<T>::from(-1.0e4f);
  v[off] = Store<T>::from(0.0f);
}

hipError_t launch_init_dead_slot(const ikv_pool &p, hipStream_t st) {
  int HD = p.Hkv * p.D;
  int64_t n = int64_t(p.L) * HD;
  dim3 grid(unsigned(cdiv(n, 256)));
  if (p.kv_dtype == IKV_BF16)
    {
      KTimer kt_("k_init_dead_slot<uint16_t>", st);
      k_init_dead_slot<uint16_t><<<grid, 256, 0, st>>>((uint16_t *)p.k_pool, (uint16_t *)p.v_pool, p.L,
                                                        p.num_slots, HD, p.dead_slot);
    }
  else
    {
      KTimer kt_("k_init_dead_slot<float>", st);
      k_init_dead_slot<float><<<grid, 256, 0, st>>>((float *)p.k_pool, (float *)p.v_pool, p.L, p.num_slots,
                                                     HD, p.dead_slot);
    }
  return hipGetLastError();
}

// One wavefront per memory row: Enc = mean of the span rows, M = decay * M + Enc,
// then the row is divided by max(||row||, 1e-12). Lane (g, c) reads channels
// 8c .. 8c+7 of span rows g, g + G, ... (G = 512 / D rows per wave step) with
// 16-byte loads; the G row groups fold with shuffles. The span rows are read once, with
// the non-temporal hint (each load instruction covers G whole rows).
typedef unsigned int qm_u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void load8_once(const uint16_t *p, float *o) {
  const qm_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const qm_u32x4 *>(p));
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = __uint_as_float(w[i] << 16);
    o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8_once(const float *p, float *o) {
  const qm_u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const qm_u32x4 *>(p));
  const qm_u32x4 b = __builtin_nontemporal_load(reinterpret_cast<const qm_u32x4 *>(p + 4));
  const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = __uint_as_float(w[i]);
}

template <typename T, int D>
__global__ void __launch_bounds__(256) k_qm_update(const ikv_session *__restrict__ sess, int L, int Hkv,
                                                   float *__restrict__ M, const T *__restrict__ q_span,
                                                   float decay) {
  constexpr int CL = D / 8;        // lanes per span row
  constexpr int G = WAVE / CL;     // span rows per wave step
  const ikv_session s = sess[blockIdx.y];
  const int rows = L * Hkv * s.R;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const int c = lane % CL, g = lane / CL;
  const int n = s.qe - s.qs;
  float *m = M + s.mem_off + int64_t(row) * D + c * 8;
  const T *q = q_span + s.qspan_off + int64_t(row) * n * D + c * 8;
  float e[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) e[k] = 0.f;
  int tq = g;
  for (; tq + 3 * G < n; tq += 4 * G) {          // four loads in flight per lane
    float a[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u) load8_once(q + int64_t(tq + u * G) * D, a[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 8; ++k) e[k] += a[u][k];
  }
  for (; tq < n; tq += G) {
    float a[8];
    load8_once(q + int64_t(tq) * D, a);
#pragma unroll
    for (int k = 0; k < 8; ++k) e[k] += a[k];
  }
#pragma unroll
  for (int o = CL; o < WAVE; o <<= 1)
#pragma unroll
    for (int k = 0; k < 8; ++k) e[k] += __shfl_xor(e[k], o, WAVE);
  float x[8];
  float ss = 0.f;
  if (g == 0) {
    float mo[8];
    load8(m, mo);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      x[k] = decay * mo[k] + (n > 0 ? e[k] / float(n) : 0.f);
      ss += x[k] * x[k];
    }
  }
  ss = wave_sum(ss);
  const float nrm = fmaxf(sqrtf(ss), 1e-12f);
  if (g == 0) {
    *reinterpret_cast<float4 *>(m) = make_float4(x[0] / nrm, x[1] / nrm, x[2] / nrm, x[3] / nrm);
    *reinterpret_cast<float4 *>(m + 4) = make_float4(x[4] / nrm, x[5] / nrm, x[6] / nrm, x[7] / nrm);
  }
}

template <typename T>
void qm_launch(const ikv_pool &p, const ikv_session *sess_dev, dim3 grid, float *M, const void *q_span, float decay,
               hipStream_t st) {
  if (p.D == 128)
    {
      KTimer kt_("k_qm_update<T, 128>", st);
      k_qm_update<T, 128><<<grid, 256, 0, st>>>(sess_dev, p.L, p.Hkv, M, (const T *)q_span, decay);
    }
  else
    {
      KTimer kt_("k_qm_update<T, 64>", st);
      k_qm_update<T, 64><<<grid, 256, 0, st>>>(sess_dev, p.L, p.Hkv, M, (const T *)q_span, decay);
    }
}

hipError_t launch_qm_update(const ikv_pool &p, const ikv_session *sess_dev, int B, int max_rows, float *M,
                            const void *q_span, float decay, hipStream_t st) {
  dim3 grid(unsigned(cdiv(max_rows, 4)), unsigned(B));
  if (p.kv_dtype == IKV_BF16) qm_launch<uint16_t>(p, sess_dev, grid, M, q_span, decay, st);
  else qm_launch<float>(p, sess_dev, grid, M, q_span, decay, st);
  return hipGetLastError();
}

}  // namespace ikv
