// gemm.hip -- bf16 matrix-core GEMM for gfx950: C[M][N] = A[M][K] * B[N][K]^T
// with fp32 accumulation and fused epilogues (plain store, + residual, SwiGLU,
// and the QKV projection's RoPE + KV-cache append).
//
// Design:
//  - workgroup tile BM x BN, K step 64; waves of 64 lanes each own a WM x WN
//    sub-tile computed with v_mfma_f32_32x32x16_bf16;
//  - the next K slice is fetched global -> registers while the matrix cores
//    work on the current one, then written to the other half of a double-
//    buffered LDS stage (one barrier per 64-wide K slice);
//  - fragment reads of k-step ks+1 are issued before the MFMAs of k-step ks;
//  - LDS rows are 128 bytes (64 bf16 of K); the 16-byte chunk c of row r is
//    stored at position c ^ (r & 7), which makes the fragment reads of 8
//    consecutive rows hit 8 distinct bank groups;
//  - tile order is XCD-aware: workgroup b runs on XCD b % 8, and each XCD is
//    handed a contiguous run of tiles taken in M-grouped order, so that the
//    tiles sharing an L2 also share A and B panels;
//  - small-M problems (weight streaming) split K over a second grid dimension
//    and finish in a deterministic reduce-and-epilogue kernel.
#include <algorithm>
#include <cmath>

#include "mx_device.h"
#include "mx_kernels.h"

namespace mx {

namespace {

constexpr int BK = 64;
constexpr int kGroupM = 8;

__device__ __forceinline__ void tile_coords(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nt = tiles_m * tiles_n;
  const int xcd = bid & 7, local = bid >> 3;
  const int q = nt >> 3, r = nt & 7;
  const int t = xcd * q + min(xcd, r) + local;
  const int group = kGroupM * tiles_n;
  const int gid = t / group;
  const int first_m = gid * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int in_group = t - gid * group;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Fused QKV epilogue for one rotary pair: packed columns c and c + 32 (c in the
// low 32-column block of a 64-column group) of token row t, fp32 values lo, hi.
// q and k heads are rotated (rotate-half pairing, dims d_lo and d_lo + hd/2)
// and rounded once; q goes to q_out, k and v to their slots in the pools.
__device__ __forceinline__ void qkv_pair_store(const GemmArgs& a, int t, int c, float lo, float hi) {
  const QkvEpilogue& e = a.qkv;
  const int hd = e.head_dim;
  const int head = c / hd, within = c % hd;
  const int64_t slot = (head >= e.nq) ? e.tok_slot[t] : 0;
  if (head < e.nq + e.nkv) {
    const int d_lo = 32 * (within / 64) + (within % 32);
    const float2 cs = e.rope_cs[(int64_t)t * (hd / 2) + d_lo];
    const float rlo = lo * cs.x - hi * cs.y;
    const float rhi = hi * cs.x + lo * cs.y;
    uint16_t* dst;
    if (head < e.nq) {
      dst = e.q_out + ((int64_t)t * e.nq + head) * hd;
    } else {
      const int64_t page = slot / 16;
      dst = e.k_pool + ((page * e.nkv + (head - e.nq)) * 16 + slot % 16) * hd;
    }
    dst[d_lo] = f32_to_bf16(rlo);
    dst[d_lo + hd / 2] = f32_to_bf16(rhi);
  } else {
    const int64_t page = slot / 16;
    uint16_t* dst = e.v_pool + ((page * e.nkv + (head - e.nq - e.nkv)) * hd) * 16 + slot % 16;
    dst[(int64_t)within * 16] = f32_to_bf16(lo);
    dst[(int64_t)(within + 32) * 16] = f32_to_bf16(hi);
  }
}

template <int BM, int BN, int WM, int WN, int EPI, bool SPLIT>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void gemm_kernel(GemmArgs a, int tiles_m,
                                                                           int tiles_n,
                                                                           int k_per_split) {
  constexpr int WAVES_N = BN / WN;
  constexpr int NWAVES = (BM / WM) * WAVES_N;
  constexpr int MB = WM / 32, NB = WN / 32;
  constexpr int STAGE = (BM + BN) * 128;  // bytes per LDS stage
  static_assert((EPI != EPI_SWIGLU && EPI != EPI_QKV) || NB % 2 == 0,
                "SwiGLU and the QKV epilogue need pairs of 32-column blocks");
  extern __shared__ __attribute__((aligned(16))) char smem[];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wave_m = wave / WAVES_N, wave_n = wave % WAVES_N;
  int tm, tn;
  tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kz = blockIdx.y;
  const int kbeg = kz * k_per_split;
  const int nk = k_per_split / BK;

  // Global -> register -> LDS staging.  Each thread owns NA + NB_ 16-byte
  // chunks of the stage: chunk q of the A tile is row (q * 256 + tid) / 8,
  // logical 16-byte column (tid % 8), stored at column (tid % 8) ^ (row % 8).
  constexpr int NTHREADS = NWAVES * 64;
  constexpr int NA = BM * 8 / NTHREADS, NBC = BN * 8 / NTHREADS;
  static_assert(NA * NTHREADS == BM * 8 && NBC * NTHREADS == BN * 8, "tile/thread mismatch");
  const int tid = threadIdx.x;
  const int lcol = tid & 7;
  const uint16_t* a_src[NA];
  const uint16_t* b_src[NBC];
  int a_dst[NA], b_dst[NBC];
#pragma unroll
  for (int q = 0; q < NA; q++) {
    const int row = (q * NTHREADS + tid) >> 3;
    a_src[q] = a.A + (int64_t)min(m0 + row, a.M - 1) * a.lda + kbeg + lcol * 8;
    a_dst[q] = row * 128 + ((lcol ^ (row & 7)) << 4);
  }
#pragma unroll
  for (int q = 0; q < NBC; q++) {
    const int row = (q * NTHREADS + tid) >> 3;
    b_src[q] = a.B + (int64_t)min(n0 + row, a.N - 1) * a.ldb + kbeg + lcol * 8;
    b_dst[q] = BM * 128 + row * 128 + ((lcol ^ (row & 7)) << 4);
  }
  u32x4 ra[NA], rb[NBC];
  auto gload = [&](int kt) {
#pragma unroll
    for (int q = 0; q < NA; q++) ra[q] = *reinterpret_cast<const u32x4*>(a_src[q] + kt * BK);
#pragma unroll
    for (int q = 0; q < NBC; q++) rb[q] = *reinterpret_cast<const u32x4*>(b_src[q] + kt * BK);
  };
  auto lstore = [&](int stage) {
    char* base = smem + stage * STAGE;
#pragma unroll
    for (int q = 0; q < NA; q++) *reinterpret_cast<u32x4*>(base + a_dst[q]) = ra[q];
#pragma unroll
    for (int q = 0; q < NBC; q++) *reinterpret_cast<u32x4*>(base + b_dst[q]) = rb[q];
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; i++)
#pragma unroll
    for (int j = 0; j < NB; j++)
#pragma unroll
      for (int r = 0; r < 16; r++) acc[i][j][r] = 0.f;

  const int frow = lane & 31, fk = lane >> 5;
  // fragment double buffer: the reads of k-step ks+1 are in flight while the
  // matrix cores work on k-step ks
  bf16x8 af[2][MB], bfr[2][NB];
  auto load_frags = [&](int buf, const char* sa, int ks) {
    const char* sb = sa + BM * 128;
    const int c = ks * 2 + fk;
#pragma unroll
    for (int i = 0; i < MB; i++) {
      const int row = wave_m * WM + i * 32 + frow;
      af[buf][i] = as_bf16x8(*reinterpret_cast<const u32x4*>(sa + row * 128 + ((c ^ (row & 7)) << 4)));
    }
#pragma unroll
    for (int j = 0; j < NB; j++) {
      const int row = wave_n * WN + j * 32 + frow;
      bfr[buf][j] = as_bf16x8(*reinterpret_cast<const u32x4*>(sb + row * 128 + ((c ^ (row & 7)) << 4)));
    }
  };
  gload(0);
  lstore(0);
  __syncthreads();
  load_frags(0, smem, 0);
  for (int kt = 0; kt < nk; kt++) {
    const char* sa = smem + (kt & 1) * STAGE;
    // the last iteration re-fetches its own K slice, keeping the body one block
    gload(min(kt + 1, nk - 1));
#pragma unroll
    for (int ks = 0; ks < BK / 16; ks++) {
      if (ks + 1 < BK / 16) load_frags((ks + 1) & 1, sa, ks + 1);
#pragma unroll
      for (int i = 0; i < MB; i++)
#pragma unroll
        for (int j = 0; j < NB; j++) acc[i][j] = mfma32(af[ks & 1][i], bfr[ks & 1][j], acc[i][j]);
      // issue order inside the k-step: the global fetch of the next slice (first
      // step only), the next step's fragment reads, then this step's MFMAs
      if (ks == 0) __builtin_amdgcn_sched_group_barrier(0x020, NA + NBC, 0);
      if (ks + 1 < BK / 16) __builtin_amdgcn_sched_group_barrier(0x100, MB + NB, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, MB * NB, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // buffer (kt + 1) & 1 was last read in iteration kt - 1, before the barrier
    // that closed it
    lstore((kt + 1) & 1);
    __syncthreads();
    load_frags(0, smem + ((kt + 1) & 1) * STAGE, 0);
  }

  // epilogue
  const int ccol = lane & 31, crow = 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < MB; i++) {
#pragma unroll
    for (int r = 0; r < 16; r++) {
      const int row = m0 + wave_m * WM + i * 32 + 8 * (r >> 2) + crow + (r & 3);
      if (row >= a.M) continue;
      if constexpr (SPLIT) {
#pragma unroll
        for (int j = 0; j < NB; j++) {
          const int colg = n0 + wave_n * WN + j * 32 + ccol;
          if (colg < a.N) a.partial[((int64_t)kz * a.M + row) * a.N + colg] = acc[i][j][r];
        }
      } else if constexpr (EPI == EPI_QKV) {
#pragma unroll
        for (int jp = 0; jp < NB / 2; jp++) {
          const int colg = n0 + wave_n * WN + jp * 64 + ccol;  // low block column
          if (colg >= a.N) continue;
          qkv_pair_store(a, row, colg, acc[i][2 * jp][r], acc[i][2 * jp + 1][r]);
        }
      } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int jp = 0; jp < NB / 2; jp++) {
          const int colg = n0 + wave_n * WN + jp * 64;  // first packed column of the pair
          if (colg >= a.N) continue;
          const float gt = acc[i][2 * jp][r], up = acc[i][2 * jp + 1][r];
          a.C[(int64_t)row * a.ldc + colg / 2 + ccol] = f32_to_bf16(silu(gt) * up);
        }
      } else {
#pragma unroll
        for (int j = 0; j < NB; j++) {
          const int colg = n0 + wave_n * WN + j * 32 + ccol;
          if (colg >= a.N) continue;
          float v = acc[i][j][r];
          if constexpr (EPI == EPI_RESIDUAL) v += bf16_to_f32(a.R[(int64_t)row * a.ldr + colg]);
          a.C[(int64_t)row * a.ldc + colg] = f32_to_bf16(v);
        }
      }
    }
  }
}

// Sum of the K splits in fixed order, then the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a, int ksplit) {
  const int ncols = (EPI == EPI_SWIGLU || EPI == EPI_QKV) ? a.N / 2 : a.N;
  const int64_t total = (int64_t)a.M * ncols;
  const int64_t plane = (int64_t)a.M * a.N;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int row = (int)(idx / ncols), col = (int)(idx % ncols);
    if constexpr (EPI == EPI_QKV) {
      const int c = (col / 32) * 64 + col % 32;
      const int64_t li = (int64_t)row * a.N + c, hi = li + 32;
      float lo = 0.f, hv = 0.f;
      for (int z = 0; z < ksplit; z++) {
        lo += a.partial[z * plane + li];
        hv += a.partial[z * plane + hi];
      }
      qkv_pair_store(a, row, c, lo, hv);
    } else if constexpr (EPI == EPI_SWIGLU) {
      const int fb = col / 32, w = col % 32;
      const int64_t gi = (int64_t)row * a.N + fb * 64 + w, ui = gi + 32;
      float g = 0.f, u = 0.f;
      for (int z = 0; z < ksplit; z++) {
        g += a.partial[z * plane + gi];
        u += a.partial[z * plane + ui];
      }
      a.C[(int64_t)row * a.ldc + col] = f32_to_bf16(silu(g) * u);
    } else {
      const int64_t pi = (int64_t)row * a.N + col;
      float v = 0.f;
      for (int z = 0; z < ksplit; z++) v += a.partial[z * plane + pi];
      if constexpr (EPI == EPI_RESIDUAL) v += bf16_to_f32(a.R[(int64_t)row * a.ldr + col]);
      a.C[(int64_t)row * a.ldc + col] = f32_to_bf16(v);
    }
  }
}

struct Plan {
  int cfg;     // tile shape index into kShapes
  int ksplit;
};

struct Shape {
  int BM, BN;
  double tflops;  // sustained rate of one full tile stream on the whole chip (measured)
};
// 256x256 and 128x256 run eight waves (2 per SIMD), the smaller shapes four.
constexpr Shape kShapes[] = {{256, 256, 1150.0}, {128, 256, 950.0}, {128, 128, 800.0},
                             {64, 128, 420.0}};
constexpr int kNumShapes = 4;

// Estimated time of each (tile shape, K split) choice: the busiest CU runs
// ceil(units / 256) tile-units at the shape's per-CU rate; K splits add the
// fp32 partial round trip; nothing beats streaming the weights once.
Plan choose(int M, int N, int K) {
  const double cus = 256.0, hbm = 5.0e12;
  Plan best{kNumShapes - 1, 1};
  double best_t = 1e30;
  for (int c = 0; c < kNumShapes; c++) {
    const int BM = kShapes[c].BM, BN = kShapes[c].BN;
    const double tiles = (double)((M + BM - 1) / BM) * ((N + BN - 1) / BN);
    for (int ks = 1; ks <= 8; ks *= 2) {
      if (K % (BK * ks) != 0 || K / ks < 4 * BK) break;
      if (ks > 1 && (double)ks * M * N > (double)kMaxSplitFloats) break;
      const double units = tiles * ks;
      const double rounds = std::ceil(units / cus);
      const double unit_flops = 2.0 * BM * BN * (double)(K / ks);
      const double t_mfma = rounds * unit_flops / (kShapes[c].tflops * 1e12 / cus);
      const double t_mem = 2.0 * ((double)N * K + (double)M * K) / hbm;
      const double t_red = ks > 1 ? ((double)ks * M * N * 4.0 * 2.0 + 2.0 * M * N) / hbm + 3e-6 : 0.0;
      const double t = std::max(t_mfma, t_mem) + t_red;
      if (t < best_t * 0.98) {
        best_t = t;
        best = {c, ks};
      }
    }
  }
  return best;
}

template <int BM, int BN, int WM, int WN, int EPI, bool SPLIT>
hipError_t run(const GemmArgs& a, int ksplit, hipStream_t stream) {
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  const int threads = (BM / WM) * (BN / WN) * 64;
  const size_t lds = 2 * (BM + BN) * 128;
  dim3 grid(tiles_m * tiles_n, ksplit);
  gemm_kernel<BM, BN, WM, WN, EPI, SPLIT><<<grid, threads, lds, stream>>>(a, tiles_m, tiles_n,
                                                                          a.K / ksplit);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN>
hipError_t run_shape(const GemmArgs& a, int ksplit, hipStream_t stream) {
  if (ksplit > 1) {
    hipError_t e = run<BM, BN, WM, WN, EPI_STORE, true>(a, ksplit, stream);
    if (e != hipSuccess) return e;
    const bool paired = a.epilogue == EPI_SWIGLU || a.epilogue == EPI_QKV;
    const int64_t total = (int64_t)a.M * (paired ? a.N / 2 : a.N);
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
    if (a.epilogue == EPI_QKV)
      splitk_reduce_kernel<EPI_QKV><<<blocks, 256, 0, stream>>>(a, ksplit);
    else if (a.epilogue == EPI_SWIGLU)
      splitk_reduce_kernel<EPI_SWIGLU><<<blocks, 256, 0, stream>>>(a, ksplit);
    else if (a.epilogue == EPI_RESIDUAL)
      splitk_reduce_kernel<EPI_RESIDUAL><<<blocks, 256, 0, stream>>>(a, ksplit);
    else
      splitk_reduce_kernel<EPI_STORE><<<blocks, 256, 0, stream>>>(a, ksplit);
    return hipGetLastError();
  }
  switch (a.epilogue) {
    case EPI_QKV: return run<BM, BN, WM, WN, EPI_QKV, false>(a, 1, stream);
    case EPI_SWIGLU: return run<BM, BN, WM, WN, EPI_SWIGLU, false>(a, 1, stream);
    case EPI_RESIDUAL: return run<BM, BN, WM, WN, EPI_RESIDUAL, false>(a, 1, stream);
    default: return run<BM, BN, WM, WN, EPI_STORE, false>(a, 1, stream);
  }
}

template <int BM, int BN, int WM, int WN>
hipError_t set_lds_attr() {
  const int lds = 2 * (BM + BN) * 128;
  hipError_t e;
#define MX_SET(EPI, SPLIT)                                                                  \
  e = hipFuncSetAttribute((const void*)gemm_kernel<BM, BN, WM, WN, EPI, SPLIT>,             \
                          hipFuncAttributeMaxDynamicSharedMemorySize, lds);                 \
  if (e != hipSuccess) return e;
  MX_SET(EPI_STORE, false)
  MX_SET(EPI_RESIDUAL, false)
  MX_SET(EPI_SWIGLU, false)
  MX_SET(EPI_QKV, false)
  MX_SET(EPI_STORE, true)
#undef MX_SET
  return hipSuccess;
}

}  // namespace

hipError_t gemm_init() {
  hipError_t e = set_lds_attr<256, 256, 128, 64>();
  if (e != hipSuccess) return e;
  e = set_lds_attr<128, 256, 64, 64>();
  if (e != hipSuccess) return e;
  e = set_lds_attr<128, 128, 64, 64>();
  if (e != hipSuccess) return e;
  return set_lds_attr<64, 128, 32, 64>();
}

size_t gemm_scratch_floats(int M, int N, int K) {
  const Plan p = choose(M, N, K);
  return p.ksplit > 1 ? (size_t)p.ksplit * M * N : 0;
}

hipError_t launch_gemm(const GemmArgs& a, size_t ws_floats, hipStream_t stream) {
  if (a.M == 0) return hipSuccess;
  Plan p = choose(a.M, a.N, a.K);
  if (p.ksplit > 1 && (size_t)p.ksplit * a.M * a.N > ws_floats) p.ksplit = 1;
  switch (p.cfg) {
    case 0: return run_shape<256, 256, 128, 64>(a, p.ksplit, stream);
    case 1: return run_shape<128, 256, 64, 64>(a, p.ksplit, stream);
    case 2: return run_shape<128, 128, 64, 64>(a, p.ksplit, stream);
    default: return run_shape<64, 128, 32, 64>(a, p.ksplit, stream);
  }
}

}  // namespace mx
