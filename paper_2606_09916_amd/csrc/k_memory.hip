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
    k_init_dead_slot<uint16_t><<<grid, 256, 0, st>>>((uint16_t *)p.k_pool, (uint16_t *)p.v_pool, p.L,
                                                      p.num_slots, HD, p.dead_slot);
  else
    k_init_dead_slot<float><<<grid, 256, 0, st>>>((float *)p.k_pool, (float *)p.v_pool, p.L, p.num_slots,
                                                   HD, p.dead_slot);
  return hipGetLastError();
}

// One wavefront per memory row: Enc = mean of the span rows, M = decay * M + Enc,
// then the row is divided by max(||row||, 1e-12). D is a multiple of 64, at most 256.
template <typename T>
__global__ void __launch_bounds__(256) k_qm_update(const ikv_session *__restrict__ sess, int L, int Hkv, int D,
                                                   float *__restrict__ M, const T *__restrict__ q_span,
                                                   float decay) {
  const ikv_session s = sess[blockIdx.y];
  const int rows = L * Hkv * s.R;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const int n = s.qe - s.qs;
  float *m = M + s.mem_off + int64_t(row) * D;
  const T *q = q_span + s.qspan_off + int64_t(row) * n * D;
  const int per = D >> 6;
  float x[4];
  float ss = 0.f;
  for (int k = 0; k < per; ++k) {
    const int d = lane + 64 * k;
    float e = 0.f;
    for (int t = 0; t < n; ++t) e += Store<T>::ld(q + int64_t(t) * D + d);
    if (n > 0) e /= float(n);
    x[k] = decay * m[d] + e;
    ss += x[k] * x[k];
  }
  ss = wave_sum(ss);
  const float nrm = fmaxf(sqrtf(ss), 1e-12f);
  for (int k = 0; k < per; ++k) m[lane + 64 * k] = x[k] / nrm;
}

hipError_t launch_qm_update(const ikv_pool &p, const ikv_session *sess_dev, int B, int max_rows, float *M,
                            const void *q_span, float decay, hipStream_t st) {
  dim3 grid(unsigned(cdiv(max_rows, 4)), unsigned(B));
  if (p.kv_dtype == IKV_BF16)
    k_qm_update<uint16_t><<<grid, 256, 0, st>>>(sess_dev, p.L, p.Hkv, p.D, M, (const uint16_t *)q_span, decay);
  else
    k_qm_update<float><<<grid, 256, 0, st>>>(sess_dev, p.L, p.Hkv, p.D, M, (const float *)q_span, decay);
  return hipGetLastError();
}

}  // namespace ikv
