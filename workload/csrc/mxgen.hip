// mxgen.hip -- device-side bulk fill of the synthetic KV pools (input
// generation only; holds none of the layer's arithmetic).
//
// Element c of the K (V) pool, in the canonical [page][head][slot][dim]
// order, holds the bf16 value of counter c of the SplitMix64 stream `key`
// (Steele, Lea and Flood 2014):
//   z = mix64(key + (c + 1) * 0x9E3779B97F4A7C15)
//   v = float((int)(z >> 40) - 2^23) * 2^-23 * 1.7320508f  -> bf16 (round to nearest even)
// Pages whose `owned` flag is 0 are filled with bf16 NaN instead.  The pools
// are written in the page layouts the attention kernels read: K pages blocked
// by 32 dims, [page][head][dim / 32][slot][32], V pages transposed,
// [page][head][dim][slot].
#include <hip/hip_runtime.h>
#include <stdint.h>

#define MXGEN_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint16_t value_at(uint64_t key, uint64_t c) {
  const uint64_t z = mix64(key + (c + 1ull) * 0x9E3779B97F4A7C15ull);
  const int32_t u = (int32_t)(z >> 40) - 8388608;
  const float f = (float)u * 0x1p-23f;
  return to_bf16(__fmul_rn(f, 1.7320508f));
}

// one thread per (page, head, slot, 8 dims)
__global__ void fill_pool_kernel(uint16_t* k_pool, uint16_t* v_pool, int64_t pages, int nkv,
                                 int d, uint64_t key_k, uint64_t key_v, const uint8_t* owned) {
  const int64_t chunks = pages * nkv * 16 * (d / 8);
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < chunks;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e0 = idx * 8;                       // canonical element index
    const int64_t page = e0 / ((int64_t)nkv * 16 * d);
    const int64_t rem = e0 % ((int64_t)nkv * 16 * d);
    const int g = (int)(rem / (16 * d));
    const int s = (int)((rem / d) % 16);
    const int dim0 = (int)(rem % d);
    const bool ok = owned == nullptr || owned[page] != 0;
    uint16_t kv[8], vv[8];
#pragma unroll
    for (int i = 0; i < 8; i++) {
      kv[i] = ok ? value_at(key_k, (uint64_t)(e0 + i)) : (uint16_t)0x7FC0;
      vv[i] = ok ? value_at(key_v, (uint64_t)(e0 + i)) : (uint16_t)0x7FC0;
    }
    uint4 w;
    w.x = kv[0] | ((uint32_t)kv[1] << 16);
    w.y = kv[2] | ((uint32_t)kv[3] << 16);
    w.z = kv[4] | ((uint32_t)kv[5] << 16);
    w.w = kv[6] | ((uint32_t)kv[7] << 16);
    // key pages blocked by 32 dims: [d / 32][16 slots][32]
    *reinterpret_cast<uint4*>(k_pool + (page * nkv + g) * (int64_t)(16 * d) + (dim0 / 32) * 512 +
                              s * 32 + dim0 % 32) = w;
    uint16_t* vb = v_pool + (page * nkv + g) * (int64_t)(16 * d);
#pragma unroll
    for (int i = 0; i < 8; i++) vb[(dim0 + i) * 16 + s] = vv[i];
  }
}

// NaN-fill whole slots (all heads and dims) of both pools
__global__ void poison_slots_kernel(uint16_t* k_pool, uint16_t* v_pool, const int64_t* slots,
                                    int64_t n, int nkv, int d) {
  const int64_t per = (int64_t)nkv * d;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n * per;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t slot = slots[idx / per];
    const int g = (int)((idx % per) / d), e = (int)(idx % d);
    const int64_t page = slot / 16;
    const int s = (int)(slot % 16);
    k_pool[(page * nkv + g) * (int64_t)(16 * d) + (e / 32) * 512 + s * 32 + e % 32] = 0x7FC0;
    v_pool[((page * nkv + g) * d + e) * 16 + s] = 0x7FC0;
  }
}

}  // namespace

MXGEN_EXPORT int mxgen_fill_pool(uint16_t* k_pool, uint16_t* v_pool, int64_t pages, int nkv, int d,
                                 uint64_t key_k, uint64_t key_v, const uint8_t* owned,
                                 hipStream_t stream) {
  if (pages <= 0 || d % 8) return 1;
  fill_pool_kernel<<<8192, 256, 0, stream>>>(k_pool, v_pool, pages, nkv, d, key_k, key_v, owned);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

MXGEN_EXPORT int mxgen_poison_slots(uint16_t* k_pool, uint16_t* v_pool, const int64_t* slots,
                                    int64_t n, int nkv, int d, hipStream_t stream) {
  if (n <= 0) return 0;
  poison_slots_kernel<<<2048, 256, 0, stream>>>(k_pool, v_pool, slots, n, nkv, d);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
