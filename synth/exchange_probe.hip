// A timing probe, for the bench: what a per-unit exchange of row normalisers between
// every workgroup of a resident grid costs on this GPU. It computes none of the
// retention method; it measures the protocol a one-key-pass score at 64 memory rows
// would need (each workgroup owns a tile of positions, so every unit's 64 row
// normalisers combine partials from every workgroup before any tile can finish that
// unit's scores).
//
// One workgroup per CU (cooperative launch), 8 waves. Per step u (one "unit"):
//   waves 0-3 spin `work_ticks` (10 ns each) standing in for the unit's compute, then,
//     with `lag` > 0, wait for the normalisers of unit u - lag (64 stamped 64-bit words,
//     prefetched one step ahead);
//   wave 4 stores this workgroup's 64 stamped partials of unit u (device scope, fire
//     and forget) and, for the pieces of earlier units it owns (piece k of unit x: rows
//     8k .. 8k + 7, owner (37 x + 32 k) mod G), checks the partials its loads of the
//     previous step returned: all present -> combine (max) and store the normalisers;
//     else reissue the loads, blocking only when the piece is due (x + lag - 1 <= u).
// A unit's pieces have 8 distinct owners, and one owner's pieces are at least 32 units
// apart (G = 256; 16 for G = 128), so with lag <= 32 an owner holds one piece at a time. A piece's partials are checked
// two steps after they are stored at the earliest, so `lag` must be at least 3.
// With mode 0 there is no exchange at all: the spin and the barrier alone. Waits are
// bounded (`spins` polls); a wait that runs out sets bit 1 (readers) or 2 (owners) of
// *fail and goes on.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int PIECES = 8;                     // pieces per unit, 8 rows each
constexpr int ROWS = 64;
constexpr int PAD_BYTES = 96 * 1024;

__device__ __forceinline__ uint64_t now10ns() { return __builtin_amdgcn_s_memrealtime(); }
__device__ __forceinline__ uint64_t ald64(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint4 ld_dev16(const void *p) {
  uint4 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}

template <int NL>                             // NL = G / 16: 16-byte loads per lane of a piece
__global__ void __launch_bounds__(512) k_exchange_probe(uint64_t *part, uint64_t *nrm, int U, int lag, int mode,
                                                        int work_ticks, uint32_t spins, uint32_t stamp,
                                                        uint32_t *fail) {
  __shared__ float stat[2][ROWS];
  extern __shared__ char pad[];               // PAD_BYTES: one workgroup per CU, as a score pass holds
  constexpr int G = 16 * NL;
  constexpr int LPR = 64 / (ROWS / PIECES);   // lanes per row within a piece: 8
  const int wg = int(blockIdx.x);
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  if (t == 0) pad[wg & 1023] = 1;
  int fu = -1, fk = 0;                        // the owned piece whose loads are in flight
  uint4 vv[NL];
  uint64_t pre = 0;
  for (int u = 0; u < U; ++u) {
    if (wave < 4) {
      const uint64_t t0 = now10ns();
      while (now10ns() - t0 < uint64_t(work_ticks)) __builtin_amdgcn_s_sleep(1);
      if (wave == 0) stat[u & 1][lane] = float((wg * 7 + lane * 13 + u) % 1000);
      const int ur = u - lag;
      if (mode == 1 && ur >= 0) {
        uint64_t v = pre;
        uint32_t s = 0;
        while (!__all(uint32_t(v) == stamp + uint32_t(ur)) && s < spins) {
          __builtin_amdgcn_s_sleep(1);
          v = ald64(nrm + int64_t(ur) * ROWS + lane);
          ++s;
        }
        if (s >= spins && lane == 0) atomicOr(fail, 1u);
        if (ur + 1 < U) pre = ald64(nrm + int64_t(ur + 1) * ROWS + lane);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (wave != 4 || mode != 1) continue;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");      // last step's loads and stores
    auto issue = [&](int x, int k) {
      const int row = k * (ROWS / PIECES) + lane / LPR, sub = lane % LPR;
      const uint64_t *src = part + (int64_t(x) * ROWS + row) * G + sub * (2 * NL);
#pragma unroll
      for (int q = 0; q < NL; ++q) vv[q] = ld_dev16(src + 2 * q);
    };
    auto finish = [&](int x, int k) -> bool {
      bool ok = true;
      float m = -1e30f;
#pragma unroll
      for (int q = 0; q < NL; ++q) {
        ok = ok && vv[q].x == stamp + uint32_t(x) && vv[q].z == stamp + uint32_t(x);
        m = fmaxf(m, fmaxf(__uint_as_float(vv[q].y), __uint_as_float(vv[q].w)));
      }
      if (!__all(ok)) return false;
#pragma unroll
      for (int o = 1; o < LPR; o <<= 1) m = fmaxf(m, __shfl_xor(m, o));
      if (lane % LPR == 0)
        __hip_atomic_store(nrm + int64_t(x) * ROWS + k * (ROWS / PIECES) + lane / LPR,
                           (uint64_t(__float_as_uint(m)) << 32) | uint32_t(stamp + x), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      return true;
    };
    if (fu >= 0) {
      const bool due = fu + lag - 1 <= u;
      bool done = finish(fu, fk);
      uint32_t s = 0;
      while (!done && due && s < spins) {                  // due: retry until every partial is in
        __builtin_amdgcn_s_sleep(1);
        issue(fu, fk);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        done = finish(fu, fk);
        ++s;
      }
      if (!done && due && lane == 0) atomicOr(fail, 2u);
      if (done || due) fu = -1;
    }
    const uint64_t v = (uint64_t(__float_as_uint(stat[u & 1][lane])) << 32) | uint32_t(stamp + u);
    __hip_atomic_store(part + (int64_t(u) * ROWS + lane) * G + wg, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (u >= 1)
#pragma unroll
      for (int k = 0; k < PIECES; ++k)
        if (((u - 1) * 37 + k * (G / PIECES)) % G == wg) {
          if (fu >= 0 && lane == 0) atomicOr(fail, 4u);    // cannot happen for lag <= 32
          fu = u - 1;
          fk = k;
        }
    if (fu >= 0) issue(fu, fk);
  }
}

}  // namespace

// Run the probe: U steps on a resident grid of G workgroups (128 or 256, at most the
// device's CUs; the launch fails otherwise), `lag` (3 to 32) steps between a unit's
// partials and the wait for its normalisers (mode 1), `work_ns` of spin per step. part: device, U * 64 * G words;
// nrm: device, U * 64 words, holding no word stamped in [stamp, stamp + U) on entry;
// fail: device word, zeroed by the caller. Returns a hipError_t value.
extern "C" int synth_exchange_probe(void *part, void *nrm, int G, int U, int lag, int mode, int work_ns,
                                    uint32_t spins, uint32_t stamp, uint32_t *fail, void *stream) {
  if (!part || !nrm || !fail || (G != 128 && G != 256) || U < 1 || (mode != 0 && mode != 1) || work_ns < 0 ||
      (mode == 1 && (lag < 3 || lag > 32)))
    return int(hipErrorInvalidValue);
  const void *kern = G == 256 ? reinterpret_cast<const void *>(k_exchange_probe<16>)
                              : reinterpret_cast<const void *>(k_exchange_probe<8>);
  hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, PAD_BYTES);
  if (e != hipSuccess) return int(e);
  int ticks = work_ns / 10;
  void *args[] = {&part, &nrm, &U, &lag, &mode, &ticks, &spins, &stamp, &fail};
  e = hipLaunchCooperativeKernel(kern, dim3(unsigned(G)), dim3(512), args, PAD_BYTES, (hipStream_t)stream);
  if (e != hipSuccess) return int(e);
  return int(hipGetLastError());
}
