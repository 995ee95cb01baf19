// A plain read of gathered pool rows, for the bench: the bytes a slot-map decode must
// move (every live slot's key and value rows of every layer), read in the same pieces
// and reduced to one word per workgroup, with nothing else computed. Its rate is the
// practical ceiling that decode attention's HBM rate is compared against. It computes
// none of the retention method.
//
// Workgroup (split, l * groups + g) reads, for the live slots [k0, k1) of its split, the
// piece of `hpw` adjacent KV heads (hpw * D * 2 bytes) of layer l's key row and value row.
// 256 threads; each 16-byte chunk of a piece is one lane's load, with the non-temporal
// hint (the faster policy for a read-once stream: 6.4-6.8 against 5.7-5.9 TB/s without it
// on the Qwen3-8B 32k live rows); eight loads per lane are in flight per round.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) k_read_ceiling(const uint4 *__restrict__ kpool, const uint4 *__restrict__ vpool,
                                                      int64_t num_slots, int Hkv, int D, int hpw,
                                                      const int32_t *__restrict__ live, int n, uint32_t *out) {
  const int groups = Hkv / hpw;
  const int l = blockIdx.y / groups, g = blockIdx.y - l * groups;
  const int nsplit = gridDim.x, split = blockIdx.x;
  const int chunk = (n + nsplit - 1) / nsplit;
  const int k0 = min(n, split * chunk), k1 = min(n, k0 + chunk);
  const int cpp = hpw * D / 8;                    // 16-byte chunks per piece
  const int64_t row_chunks = int64_t(Hkv) * D / 8;
  const int64_t base = int64_t(l) * num_slots * row_chunks + int64_t(g) * cpp;
  const int total = (k1 - k0) * cpp;              // chunks of this split, keys (values alike)
  uint32_t acc = 0;
  for (int i0 = int(threadIdx.x); i0 < total; i0 += 8 * 256) {
    uint4 a[8], b[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int i = i0 + r * 256;
      if (i < total) {
        const int k = k0 + i / cpp, c = i - (i / cpp) * cpp;
        const int64_t off = base + int64_t(live[k]) * row_chunks + c;
        const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(kpool + off));
        const u32x4 y = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(vpool + off));
        a[r] = make_uint4(x.x, x.y, x.z, x.w);
        b[r] = make_uint4(y.x, y.y, y.z, y.w);
      } else {
        a[r] = b[r] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) acc ^= a[r].x ^ a[r].y ^ a[r].z ^ a[r].w ^ b[r].x ^ b[r].y ^ b[r].z ^ b[r].w;
  }
  __shared__ uint32_t red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t x = 0;
    for (int i = 0; i < 256; ++i) x ^= red[i];
    out[blockIdx.y * nsplit + split] = x;
  }
}

}  // namespace

// Read the key and value rows of the n live slots (device int32, each in [0, num_slots))
// of every layer of bf16 pools [L][num_slots][Hkv][D], in pieces of hpw adjacent heads
// (Hkv a multiple of hpw, D a multiple of 8), `splits` workgroups per (layer, head
// group). `out` (device) receives splits * L * Hkv / hpw words. Returns a hipError_t
// value (0 on success); asynchronous on `stream`.
extern "C" int synth_read_ceiling(const void *kpool, const void *vpool, int L, int64_t num_slots, int Hkv, int D,
                                  int hpw, const int32_t *live, int n, int splits, uint32_t *out, void *stream) {
  if (!kpool || !vpool || !live || !out || L < 1 || Hkv < 1 || hpw < 1 || Hkv % hpw || D < 8 || D % 8 ||
      num_slots < 1 || n < 0 || splits < 1 || int64_t(L) * (Hkv / hpw) > 65535 ||
      ((reinterpret_cast<uintptr_t>(kpool) | reinterpret_cast<uintptr_t>(vpool)) & 15))
    return int(hipErrorInvalidValue);
  if (int64_t(n) * hpw * D / 8 >= (int64_t(1) << 31)) return int(hipErrorInvalidValue);
  k_read_ceiling<<<dim3(unsigned(splits), unsigned(L * (Hkv / hpw))), 256, 0, (hipStream_t)stream>>>(
      static_cast<const uint4 *>(kpool), static_cast<const uint4 *>(vpool), num_slots, Hkv, D, hpw, live, n, out);
  return int(hipGetLastError());
}
