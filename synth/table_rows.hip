// Pool rows drawn from a table, on the GPU: the input generator of workloads too
// large to draw on the host (the batched one-GPU share holds about 219 GB of keys and
// values). It computes none of the retention method.
//
// Row (l, slot, h) of a pool [L][num_slots][Hkv][D] is the window
//   table[o .. o + D),  o = splitmix64(key + (r + 1) * GAMMA) >> (64 - log2_T),
//   r = (l * num_slots + slot) * Hkv + h,
// of a table of T + D bfloat16 values (T = 2^log2_T). splitmix64 is the output
// function of SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
// generators", OOPSLA 2014). The host side of the generator (synth.table_rows)
// computes the same offsets with numpy and gathers the same windows.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t splitmix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// One thread per 8 elements of a row, layer blockIdx.y: grid-stride over (k, h, chunk)
// within the layer (32-bit: the host checks n_slots * Hkv * D / 8 < 2^31), where k
// indexes `slots` (or is the slot itself when slots is NULL).
__global__ void k_table_rows(uint16_t *__restrict__ pool, int64_t num_slots, int Hkv, int D,
                             const int32_t *__restrict__ slots, int64_t n_slots, const uint16_t *__restrict__ table,
                             int log2_T, uint64_t key) {
  const int l = blockIdx.y;
  const uint32_t chunks = uint32_t(D / 8);
  const uint32_t total = uint32_t(n_slots) * uint32_t(Hkv) * chunks;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const uint32_t c = i % chunks, q = i / chunks;
    const uint32_t h = q % uint32_t(Hkv), k = q / uint32_t(Hkv);
    const int64_t slot = slots ? int64_t(slots[k]) : int64_t(k);
    const uint64_t r = (uint64_t(l) * uint64_t(num_slots) + uint64_t(slot)) * uint64_t(Hkv) + h;
    const uint64_t o = splitmix64(key + (r + 1) * GAMMA) >> (64 - log2_T);
    const uint16_t *src = table + o + 8 * c;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = uint32_t(src[2 * e]) | (uint32_t(src[2 * e + 1]) << 16);
    uint16_t *dst = pool + ((int64_t(l) * num_slots + slot) * Hkv + h) * D + 8 * c;
    *reinterpret_cast<uint4 *>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

}  // namespace

// Fill rows of a bf16 pool [L][num_slots][Hkv][D] from `table` (device, T + D values,
// T = 2^log2_T): every slot when `slots` is NULL (then n_slots = num_slots), else the
// n_slots listed slots (device int32, each in [0, num_slots)). D a multiple of 8, pool
// 16-byte aligned. Returns a hipError_t value (0 on success); asynchronous on `stream`.
extern "C" int synth_table_rows(void *pool, int L, int64_t num_slots, int Hkv, int D, const int32_t *slots,
                                int64_t n_slots, const void *table, int log2_T, uint64_t key, void *stream) {
  if (!pool || !table || L < 1 || Hkv < 1 || D < 8 || D % 8 || num_slots < 1 || n_slots < 0 || log2_T < 1 ||
      log2_T > 40 || (!slots && n_slots != num_slots) || (reinterpret_cast<uintptr_t>(pool) & 15))
    return int(hipErrorInvalidValue);
  if (n_slots == 0) return 0;
  const int64_t per_layer = n_slots * Hkv * (D / 8);
  if (per_layer >= (int64_t(1) << 31) || L > 65535) return int(hipErrorInvalidValue);
  const int64_t blocks = (per_layer + 255) / 256;
  k_table_rows<<<dim3(unsigned(blocks < 16384 ? blocks : 16384), unsigned(L)), 256, 0, (hipStream_t)stream>>>(
      static_cast<uint16_t *>(pool), num_slots, Hkv, D, slots, n_slots, static_cast<const uint16_t *>(table), log2_T,
      key);
  return int(hipGetLastError());
}
