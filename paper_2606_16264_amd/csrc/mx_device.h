// mx_device.h -- device-side types and helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mx {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

#define MX_LDS __attribute__((address_space(3)))

// Activations that feed a projection (the RMSNorm outputs, the attention
// output, the SwiGLU output) are stored in the GEMM operand tile layout: an
// M x K matrix as ceil(M / 16) tile rows of K / 32 tiles, each 16-row x
// 32-column tile one contiguous kilobyte (K a multiple of 32), like the packed
// weights.  A GEMM copy instruction then reads one whole kilobyte instead of
// sixteen 64-byte row pieces.  Each tile row is followed by one unused tile:
// without it the tile rows of a large K lie a power of two apart (256 KB at
// K = 8192), the sixteen tiles of rows that one K slice of a 256-row GEMM tile
// reads share their L2 sets, and the 70B-shaped gate/up projection missed L2
// for 19.4 GB per launch instead of 12.8 GB (and ran 2% slower).
__host__ __device__ __forceinline__ int64_t tile_row_pitch(int64_t K) { return 16 * K + 512; }
// Element offset of (row r, column c):
__host__ __device__ __forceinline__ int64_t tile_index(int64_t r, int64_t c, int64_t K) {
  return (r >> 4) * tile_row_pitch(K) + (c >> 5) * 512 + (r & 15) * 32 + (c & 31);
}
// Elements of an M x K matrix in the tile layout (whole tile rows).
__host__ __device__ __forceinline__ int64_t tile_elems(int64_t M, int64_t K) {
  return (M + 15) / 16 * tile_row_pitch(K);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// Round-to-nearest-even float -> bf16 bits; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two floats to a pair of bf16 (lo in the low half), round-to-nearest-even
// like f32_to_bf16: one v_cvt_pk_bf16_f32 (the conversion written per
// element became two conversions, a shift and an or).
typedef __bf16 mx_bf16x2 __attribute__((ext_vector_type(2)));
typedef float mx_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const mx_f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, mx_bf16x2));
}

// 16x16x32 bf16 matrix-core product, fp32 accumulate.
// A: lane l holds row (l % 16), k = 8 * (l / 16) .. +7
// B: lane l holds col (l % 16), k = 8 * (l / 16) .. +7
// C: lane l holds col (l % 16), rows 4 * (l / 16) .. +3
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Hand-placed waits and LDS traffic for kernels that copy global -> LDS with
// the DMA path (global_load_lds, 16 bytes per lane; the hardware tracks it with
// vmcnt only) and read their matrix-core fragments with ds_read_b128 issued
// from inline assembly, so that every wait is placed by hand rather than
// inferred (the compiler would otherwise wait for all DMA in flight before any
// LDS read).  The compiler takes an inline-assembly read's result as available
// at once: pin() ties fragment registers to the preceding wait so that no
// consumer is scheduled above it, and the registers must stay live until then.
template <int N>
__device__ __forceinline__ void lgkm_wait() {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N) : "memory");
}
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }
template <int K>
__device__ __forceinline__ void pin(u32x4 (&f)[K]) {
#pragma unroll
  for (int i = 0; i < K; i++) asm volatile("" : "+v"(f[i]));
}
__device__ __forceinline__ u32x4 lds_read16(unsigned addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}
// the same with a constant byte offset added by the instruction
template <int OFF>
__device__ __forceinline__ u32x4 lds_read16_at(unsigned addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
  return v;
}
__device__ __forceinline__ void dma16(const void* g, unsigned lds_addr) {
  __builtin_amdgcn_global_load_lds(g, (MX_LDS void*)(size_t)lds_addr, 16, 0, 0);
}

// Request record uploaded by the host planner.
struct ReqDev {
  int32_t tok_start;  // first row of the request in the batch
  int32_t n_new;
  int32_t ctx_len;
  int32_t kv_len;     // ctx_len + n_new
  int32_t page_start; // offset of the page table in the flat page array
  int32_t n_pages;    // pages the request actually uses: ceil(kv_len / 16)
  int32_t phase;
  int32_t n_split;    // decode: number of key splits (1 = no merge)
};

// Attention work item (16 bytes).
//   kind 0 (decode): q heads [head, head + nrows) of the request's single token,
//                    pages [start, start + split_pages) of its table; part =
//                    split index (ignored when the request has one split).
//   kind 1 (prefill): q head `head`, query rows [start, start + kPrefillTileRows)
//                     of the request.
constexpr int kPrefillTileRows = 128;  // four waves x two blocks of 16 rows
struct AttnItem {
  int32_t req;
  int16_t head;
  int8_t kind;
  int8_t nrows;
  int32_t start;
  int32_t part;
};

struct MergeItem {
  int32_t req;
  int32_t part_base;  // partial index of (req, q head 0, split 0)
};

}  // namespace mx
