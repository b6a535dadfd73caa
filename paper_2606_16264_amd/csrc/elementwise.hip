// elementwise.hip -- the memory-bound kernels of the layer step on gfx950:
// token map + rotary table, RMSNorm, KV append, gather, weight packing.
#include <algorithm>

#include "mx_device.h"
#include "mx_kernels.h"

namespace mx {

namespace {

// ---------------------------------------------------------------- token map
// One thread per (token, rotary pair).  The token's request is found by binary
// search over the requests' first rows (copied to LDS first when they fit, so
// that the search does not chain global-memory round trips); token
// t = tok_start + i of request r sits at position ctx_len + i and writes slot
// page * 16 + pos % 16.  The rotary angle pos * theta^(-2i/d) is formed and
// reduced modulo 2 pi in double precision; its cosine and sine are then taken
// in single precision.
constexpr int kLdsReqs = 4096;

struct TokenMapArgs {
  const ReqDev* reqs;
  int R, T;
  const int32_t* pages;
  int32_t* tok_req;
  int32_t* tok_pos;
  int64_t* tok_slot;
  const double* inv_freq;
  float2* rope_cs;
  int half;
};

// Block-uniform: every thread of the block calls it (it synchronises the block).
__device__ __forceinline__ void token_map_block(const TokenMapArgs& a, int block, int* s_start) {
  const bool in_lds = a.R <= kLdsReqs;
  if (in_lds) {
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) s_start[r] = a.reqs[r].tok_start;
    __syncthreads();
  }
  const int64_t idx = (int64_t)block * blockDim.x + threadIdx.x;
  const int t = (int)(idx / a.half), i = (int)(idx % a.half);
  if (t >= a.T) return;
  int lo = 0, hi = a.R - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    const int start = in_lds ? s_start[mid] : a.reqs[mid].tok_start;
    if (start <= t) lo = mid; else hi = mid - 1;
  }
  const ReqDev rq = a.reqs[lo];
  const int pos = rq.ctx_len + (t - rq.tok_start);
  if (i == 0) {
    const int64_t page = a.pages[rq.page_start + pos / 16];
    a.tok_req[t] = lo;
    a.tok_pos[t] = pos;
    a.tok_slot[t] = page * 16 + pos % 16;
  }
  if (a.rope_cs) {
    const double ang = (double)pos * a.inv_freq[i];
    const double two_pi = 6.283185307179586476925286766559;
    const double r = ang - rint(ang / two_pi) * two_pi;
    float sn, cs;
    sincosf((float)r, &sn, &cs);
    a.rope_cs[(int64_t)t * a.half + i] = make_float2(cs, sn);
  }
}

__global__ __launch_bounds__(256) void token_map_kernel(TokenMapArgs a) {
  __shared__ int s_start[kLdsReqs];
  token_map_block(a, blockIdx.x, s_start);
}

// ---------------------------------------------------------------- RMSNorm
// Two rows per block of 256 threads, written in the tile layout.  Thread t
// works on row 2j + (t / 4) % 2 and on its chunks (8 columns each)
// i = 4 (t / 8) + t % 4 + 128 k: the eight threads 8 s .. 8 s + 7 hold the same
// 32 columns of both rows, which are one 128-byte line of a 16 x 32 tile
// (rows 2j and 2j + 1 are adjacent in it), so every store instruction writes
// whole lines (70B-shaped norms: 59-65 us; 70-77 us with one row per block,
// whose stores covered half a line each).  Rows of up to 8192
// elements are held in registers between the sum of squares and the scaling
// (with the gains, read in the same first pass), so a row is read from memory
// once; longer rows are read twice.
constexpr int kPairChunks = 8;  // 16-byte chunks per thread held in registers

__device__ __forceinline__ void rms_scale_store(u32x4 v, u32x4 gv, float inv, u32x4* dst) {
  u32x4 w;
#pragma unroll
  for (int j = 0; j < 4; j++) {
    const float a = __uint_as_float(v[j] << 16) * inv * __uint_as_float(gv[j] << 16);
    const float b = __uint_as_float(v[j] & 0xFFFF0000u) * inv * __uint_as_float(gv[j] & 0xFFFF0000u);
    w[j] = pack_bf16x2(a, b);
  }
  *dst = w;
}

__device__ __forceinline__ float sum_squares(u32x4 v) {
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < 4; j++) {
    const float a = __uint_as_float(v[j] << 16), b = __uint_as_float(v[j] & 0xFFFF0000u);
    ss += a * a + b * b;
  }
  return ss;
}

// Sum over the block's threads of one row (par = (t / 4) % 2); red holds 8 floats.
__device__ __forceinline__ float pair_sum_256(float v, float* red, int par) {
  // every lane offset but 4, which would cross to the other row
  v += __shfl_xor(v, 1);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 8);
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0 || lane == 4) red[2 * wave + (lane >> 2)] = v;
  __syncthreads();
  return red[par] + red[2 + par] + red[4 + par] + red[6 + par];
}

__device__ __forceinline__ void rmsnorm_pair(const uint16_t* __restrict__ x,
                                             const uint16_t* __restrict__ g,
                                             uint16_t* __restrict__ out, int H, float eps,
                                             int64_t pair, int64_t T, float* red) {
  const int t = threadIdx.x;
  const int par = (t >> 2) & 1;
  const int64_t row = 2 * pair + par;
  const bool live = row < T;  // the second row of the last pair may not exist
  const int i0 = 4 * (t >> 3) + (t & 3);
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + (live ? row : 2 * pair) * H);
  const u32x4* gr = reinterpret_cast<const u32x4*>(g);
  auto outc = [&](int c) { return reinterpret_cast<u32x4*>(out + tile_index(row, 8 * c, H)); };
  const int nchunk = H / 8;
  if (nchunk <= kPairChunks * 128) {
    u32x4 v[kPairChunks], gv[kPairChunks];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < kPairChunks; k++) {
      const int c = i0 + k * 128;
      v[k] = live && c < nchunk ? xr[c] : u32x4{0, 0, 0, 0};
      gv[k] = c < nchunk ? gr[c] : u32x4{0, 0, 0, 0};
      ss += sum_squares(v[k]);
    }
    const float inv = 1.0f / sqrtf(pair_sum_256(ss, red, par) / (float)H + eps);
#pragma unroll
    for (int k = 0; k < kPairChunks; k++) {
      const int c = i0 + k * 128;
      if (live && c < nchunk) rms_scale_store(v[k], gv[k], inv, outc(c));
    }
    return;
  }
  float ss = 0.f;
  if (live)
    for (int c = i0; c < nchunk; c += 128) ss += sum_squares(xr[c]);
  const float inv = 1.0f / sqrtf(pair_sum_256(ss, red, par) / (float)H + eps);
  if (live)
    for (int c = i0; c < nchunk; c += 128) rms_scale_store(xr[c], gr[c], inv, outc(c));
}

// The split-K reduce of a residual GEMM fused with the RMSNorm of its output,
// one row per block of 512 threads: x1 = bf16(sum_z partial[z] + R), the sums
// taken in split order and then the residual, exactly as the stand-alone
// reduce does, and h = RMSNorm(x1, g) from the rounded x1, exactly as
// rmsnorm_pair does; the row stays in registers between the two (rows of up to
// kFusedNormMaxH elements).  Every plane's loads of a thread (up to
// kNormPlanes of them) are issued before the first sum, so that the planes
// cost one memory round trip, not one each; further planes are summed one by
// one.

__global__ __launch_bounds__(kNormThreads) void reduce_residual_rmsnorm_kernel(
    const float* __restrict__ partial, int ksplit, const uint16_t* __restrict__ R,
    uint16_t* __restrict__ x1, const uint16_t* __restrict__ g, uint16_t* __restrict__ h,
    int row0, int rows, int H, float eps) {
  // block b: row row0 + b of R, x1 and h; row b of the planes ([rows][H] each)
  __shared__ float red[kNormThreads / 64];
  const int64_t row = row0 + (int64_t)blockIdx.x;
  const int nchunk = H / 8;
  const u32x4* gr = reinterpret_cast<const u32x4*>(g);
  u32x4* xrow = reinterpret_cast<u32x4*>(x1 + row * H);
  u32x4 gv[kNormChunks], v[kNormChunks];
  const int64_t plane4 = (int64_t)rows * H / 4;  // one plane in f32x4
  const f32x4* prow = reinterpret_cast<const f32x4*>(partial + (int64_t)blockIdx.x * H);
  const u32x4* rrow = reinterpret_cast<const u32x4*>(R + row * H);
  f32x4 pl[kNormChunks][kNormPlanes][2];
  u32x4 r[kNormChunks];
#pragma unroll
  for (int k = 0; k < kNormChunks; k++) {
    const int c = threadIdx.x + k * kNormThreads;
    const bool in = c < nchunk;
#pragma unroll
    for (int z = 0; z < kNormPlanes; z++) {
      if (in && z < ksplit) {
        pl[k][z][0] = prow[z * plane4 + 2 * c];
        pl[k][z][1] = prow[z * plane4 + 2 * c + 1];
      }
    }
    r[k] = in ? rrow[c] : u32x4{0, 0, 0, 0};
    gv[k] = in ? gr[c] : u32x4{0, 0, 0, 0};
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kNormChunks; k++) {
    const int c = threadIdx.x + k * kNormThreads;
    v[k] = u32x4{0, 0, 0, 0};
    if (c >= nchunk) continue;
    f32x4 lo = pl[k][0][0], hi = pl[k][0][1];
#pragma unroll
    for (int z = 1; z < kNormPlanes; z++) {
      if (z < ksplit) {
#pragma unroll
        for (int j = 0; j < 4; j++) {
          lo[j] += pl[k][z][0][j];
          hi[j] += pl[k][z][1][j];
        }
      }
    }
    for (int z = kNormPlanes; z < ksplit; z++) {
      const f32x4 plo = prow[z * plane4 + 2 * c], phi = prow[z * plane4 + 2 * c + 1];
#pragma unroll
      for (int j = 0; j < 4; j++) {
        lo[j] += plo[j];
        hi[j] += phi[j];
      }
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      v[k][j] = pack_bf16x2(lo[2 * j] + __uint_as_float(r[k][j] << 16),
                            lo[2 * j + 1] + __uint_as_float(r[k][j] & 0xFFFF0000u));
      v[k][2 + j] = pack_bf16x2(hi[2 * j] + __uint_as_float(r[k][2 + j] << 16),
                                hi[2 * j + 1] + __uint_as_float(r[k][2 + j] & 0xFFFF0000u));
    }
    xrow[c] = v[k];
    ss += sum_squares(v[k]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; w++) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int k = 0; k < kNormChunks; k++) {
    const int c = threadIdx.x + k * kNormThreads;
    // h in the tile layout, like rmsnorm_pair's output (one row per block: each
    // store covers half a line; this kernel runs on the split rows only)
    if (c < nchunk)
      rms_scale_store(v[k], gv[k], inv, reinterpret_cast<u32x4*>(h + tile_index(row, 8 * c, H)));
  }
}

__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t* __restrict__ x,
                                                      const uint16_t* __restrict__ g,
                                                      uint16_t* __restrict__ out, int T, int H,
                                                      float eps) {
  __shared__ float red[8];
  rmsnorm_pair(x, g, out, H, eps, blockIdx.x, T, red);
}

// The first kernel of a layer step: the token map (blocks 0 .. map_blocks - 1)
// and the first RMSNorm (one block per pair of rows after them), which do not
// depend on each other, in one launch.
__global__ __launch_bounds__(256) void prologue_kernel(TokenMapArgs a, int map_blocks,
                                                       const uint16_t* __restrict__ x,
                                                       const uint16_t* __restrict__ g,
                                                       uint16_t* __restrict__ out, int H,
                                                       float eps) {
  __shared__ int s_start[kLdsReqs];
  if ((int)blockIdx.x < map_blocks)
    token_map_block(a, blockIdx.x, s_start);
  else
    rmsnorm_pair(x, g, out, H, eps, (int64_t)blockIdx.x - map_blocks, a.T,
                 reinterpret_cast<float*>(s_start));
}

// ---------------------------------------------------------------- KV append
__global__ __launch_bounds__(256) void kv_append_kernel(const uint16_t* __restrict__ k_new,
                                                        const uint16_t* __restrict__ v_new,
                                                        uint16_t* __restrict__ k_pool,
                                                        uint16_t* __restrict__ v_pool,
                                                        const int64_t* __restrict__ tok_slot,
                                                        int nkv, int d) {
  const int64_t t = blockIdx.x;
  const int64_t slot = tok_slot[t];
  const int64_t page = slot / 16;
  const int s_in = (int)(slot % 16);
  const int n = nkv * d;
  const uint16_t* ks = k_new + t * n;
  const uint16_t* vs = v_new + t * n;
  // keys: 16-byte chunks; a key page is blocked by 32 dims, [d / 32][16][32]
  for (int c = threadIdx.x; c < n / 8; c += blockDim.x) {
    const int g = (c * 8) / d, e = (c * 8) % d;
    *reinterpret_cast<u32x4*>(k_pool + (page * nkv + g) * 16 * d + (e / 32) * 512 + s_in * 32 +
                              e % 32) = *reinterpret_cast<const u32x4*>(ks + c * 8);
  }
  for (int u = threadIdx.x; u < n; u += blockDim.x) {
    const int g = u / d, e = u % d;
    v_pool[((page * nkv + g) * d + e) * 16 + s_in] = vs[u];
  }
}

// ---------------------------------------------------------------- gather
__global__ __launch_bounds__(256) void gather_kernel(const uint16_t* __restrict__ k_pool,
                                                     const uint16_t* __restrict__ v_pool,
                                                     const int32_t* __restrict__ pages, int nkv,
                                                     int d, uint16_t* __restrict__ k_out,
                                                     uint16_t* __restrict__ v_out) {
  const int64_t j = blockIdx.x;
  const int64_t page = pages[j / 16];
  const int s_in = (int)(j % 16);
  const int n = nkv * d;
  for (int u = threadIdx.x; u < n; u += blockDim.x) {
    const int g = u / d, e = u % d;
    k_out[j * n + u] = k_pool[(page * nkv + g) * 16 * d + (e / 32) * 512 + s_in * 32 + e % 32];
    v_out[j * n + u] = v_pool[((page * nkv + g) * d + e) * 16 + s_in];
  }
}

// ---------------------------------------------------------------- weight packing
// Packed row n of a weight matrix -> its source row.  kind 1 (w_qkv): rows
// of q and k heads with head_dim 128 are permuted within the head so that
// packed rows 64 g + w and 64 g + 32 + w hold dims 32 g + w and 64 + 32 g + w
// (the two halves of a rotary pair); v rows and head_dim 64 keep their order.
// kind 2 (w_gate_up): block b = n / 32; even blocks are gate rows, odd blocks
// the up rows of the same 32 features.  kind 0: identity.
__device__ __forceinline__ int packed_source_row(int n, int kind, int nq, int nkv, int d, int F) {
  if (kind == 1) {
    const int head = n / d, within = n % d;
    int sw = within;
    if (head < nq + nkv && d == 128) {
      const int g = within / 64, blk = (within % 64) / 32, w = within % 32;
      sw = blk * 64 + g * 32 + w;
    }
    return head * d + sw;
  }
  if (kind == 2) {
    const int b = n / 32, w = n % 32, fb = b / 2;
    return (b % 2 == 0) ? fb * 32 + w : F + fb * 32 + w;
  }
  return n;
}

// One workgroup per 16-row block: 16-byte pieces in destination order (piece
// q of row r of k-chunk kc), so that the stores are contiguous.
__global__ __launch_bounds__(256) void pack_tiled_kernel(const uint16_t* __restrict__ src,
                                                         uint16_t* __restrict__ dst, int K,
                                                         int kind, int nq, int nkv, int d, int F) {
  const int nb = blockIdx.x;
  const int pieces = (K / 32) * 16 * 4;
  u32x4* o = reinterpret_cast<u32x4*>(dst + (int64_t)nb * 16 * K);
  for (int p = threadIdx.x; p < pieces; p += blockDim.x) {
    const int q = p & 3, r = (p >> 2) & 15, kc = p >> 6;
    const int srow = packed_source_row(nb * 16 + r, kind, nq, nkv, d, F);
    o[p] = *reinterpret_cast<const u32x4*>(src + (int64_t)srow * K + kc * 32 + q * 8);
  }
}

// Metadata upload: 16-byte words from the pinned host staging buffer (read
// through its device mapping) into the workspace.
__global__ __launch_bounds__(256) void upload_kernel(const u32x4* __restrict__ src,
                                                     u32x4* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

}  // namespace

hipError_t launch_upload(const void* host_mapped, void* dst, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  if (bytes % 16 != 0 || (size_t)host_mapped % 16 != 0 || (size_t)dst % 16 != 0)
    return hipErrorInvalidValue;
  const int64_t n = (int64_t)(bytes / 16);
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 1024);
  upload_kernel<<<blocks, 256, 0, stream>>>(static_cast<const u32x4*>(host_mapped),
                                            static_cast<u32x4*>(dst), n);
  return hipGetLastError();
}

hipError_t launch_token_map(const ReqDev* reqs, int R, int T, const int32_t* pages,
                            int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot,
                            const double* inv_freq, float2* rope_cs, int half,
                            hipStream_t stream) {
  if (R == 0 || T == 0) return hipSuccess;
  if (!rope_cs) half = 1;
  const int64_t n = (int64_t)T * half;
  const TokenMapArgs a{reqs, R, T, pages, tok_req, tok_pos, tok_slot, inv_freq, rope_cs, half};
  token_map_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(a);
  return hipGetLastError();
}

hipError_t launch_prologue(const ReqDev* reqs, int R, int T, const int32_t* pages,
                           int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot,
                           const double* inv_freq, float2* rope_cs, int half,
                           const uint16_t* x, const uint16_t* g, uint16_t* out, int H, float eps,
                           hipStream_t stream) {
  if (R == 0 || T == 0) return hipSuccess;
  const int64_t map_blocks = ((int64_t)T * half + 255) / 256;
  const TokenMapArgs a{reqs, R, T, pages, tok_req, tok_pos, tok_slot, inv_freq, rope_cs, half};
  prologue_kernel<<<(unsigned)(map_blocks + (T + 1) / 2), 256, 0, stream>>>(a, (int)map_blocks, x,
                                                                            g, out, H, eps);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* g, uint16_t* out, int T, int H,
                          float eps, hipStream_t stream) {
  if (T == 0) return hipSuccess;
  rmsnorm_kernel<<<(T + 1) / 2, 256, 0, stream>>>(x, g, out, T, H, eps);
  return hipGetLastError();
}

hipError_t launch_reduce_residual_rmsnorm(const float* partial, int ksplit, const uint16_t* R,
                                          uint16_t* x1, const uint16_t* g, uint16_t* h, int M,
                                          int H, float eps, int split_row, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (H % 32 != 0 || H > kFusedNormMaxH || ksplit < 1 || split_row < 0 || split_row > M)
    return hipErrorInvalidValue;
  // Rows below split_row were completed by the GEMM itself (a row split of
  // the projection): they only need the RMSNorm of x1, which the plain norm
  // kernel does at its own occupancy (the fused kernel's plane registers,
  // 166 VGPRs, leave one 512-thread block per CU: as one launch the 70B
  // iteration's 8448 rows took 86 us).  The planes cover rows [split_row, M).
  if (split_row > 0) rmsnorm_kernel<<<(split_row + 1) / 2, 256, 0, stream>>>(x1, g, h, split_row, H, eps);
  const int tail = M - split_row;
  if (tail > 0)
    reduce_residual_rmsnorm_kernel<<<tail, kNormThreads, 0, stream>>>(partial, ksplit, R, x1, g, h,
                                                                      split_row, tail, H, eps);
  return hipGetLastError();
}

hipError_t launch_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                            uint16_t* v_pool, const int64_t* tok_slot, int T, int nkv, int d,
                            hipStream_t stream) {
  if (T == 0) return hipSuccess;
  kv_append_kernel<<<T, 256, 0, stream>>>(k_new, v_new, k_pool, v_pool, tok_slot, nkv, d);
  return hipGetLastError();
}

hipError_t launch_pack_tiled(const uint16_t* src, uint16_t* dst, int N, int K, int kind, int nq,
                             int nkv, int d, int F, hipStream_t stream) {
  if (N % 16 != 0 || K % 32 != 0) return hipErrorInvalidValue;
  pack_tiled_kernel<<<N / 16, 256, 0, stream>>>(src, dst, K, kind, nq, nkv, d, F);
  return hipGetLastError();
}

hipError_t launch_gather(const uint16_t* k_pool, const uint16_t* v_pool, const int32_t* pages,
                         int len, int nkv, int d, uint16_t* k_out, uint16_t* v_out,
                         hipStream_t stream) {
  if (len == 0) return hipSuccess;
  gather_kernel<<<len, 256, 0, stream>>>(k_pool, v_pool, pages, nkv, d, k_out, v_out);
  return hipGetLastError();
}

}  // namespace mx
