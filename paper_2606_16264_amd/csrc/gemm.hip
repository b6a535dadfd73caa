// gemm.hip -- bf16 matrix-core GEMM for gfx950: C[M][N] = A[M][K] * B[N][K]^T
// with fp32 accumulation and fused epilogues (plain store, + residual, SwiGLU,
// and the QKV projection's RoPE + KV-cache append).
//
// Design:
//  - workgroup tile BM x BN, K step 64; waves of 64 lanes each own a WM x WN
//    sub-tile computed with v_mfma_f32_16x16x32_bf16 (one product per 16 x 16
//    block and 32-wide K slice: under the chip's power limit it sustains a
//    higher rate than the 32 x 32 x 16 form, for the same LDS reads);
//  - K is consumed in 32-wide slices through an LDS ring (4 stages; 3 for the
//    shape that puts two workgroups on a CU) filled by the DMA path
//    (global_load_lds): the other slices are in flight while the matrix cores
//    work on one, and no registers are spent on staging;
//  - B is addressed through block, row and K-slice strides: row-major, or the
//    packed weights' 16 x 32 tiles of 1 KB, where each DMA instruction reads
//    one contiguous kilobyte;
//  - a slice runs in two phases (the two halves of the wave's A blocks against
//    all its B blocks); each phase's MFMAs are issued one at a time, with the
//    slice's DMA issues (first phase) and the next slice's fragment reads
//    (second phase) spread between them, so that a wave keeps the matrix core
//    fed while it issues its memory instructions; one barrier per slice;
//  - LDS rows are 64 bytes (32 bf16 of K); the 16-byte chunk c of row r is
//    stored at c ^ swz(r), which makes the fragment reads of 16 consecutive
//    rows hit 16 distinct bank groups (the LDS serves a 16-byte read for 16
//    lanes at a time from 64 banks);
//  - tile order is XCD-aware: workgroup b runs on XCD b % 8, and each XCD is
//    handed a contiguous run of tiles taken in M-grouped order, so that the
//    tiles sharing an L2 also share A and B panels;
//  - a K split runs over a second grid dimension (split z of S takes the
//    64-wide K chunks [z C / S, (z + 1) C / S) of the C in K, so S need not
//    divide C) and finishes in a deterministic reduce-and-epilogue kernel;
//  - a cost model picks tile shape and K split per problem (a per-CU feed
//    estimate for few rows, rounds of tile-units for more), and may run the
//    rows in two launches: the first in whole rounds of tiles, the rest as a
//    GEMM of their own (split over K), so that a problem a little over a whole
//    number of rounds does not pay for a mostly empty last round.
#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <tuple>

#include "mx_device.h"
#include "mx_kernels.h"

namespace mx {

namespace {

constexpr int BK = 64;    // K granularity of a split (and of the problem)
constexpr int BKS = 32;   // K per LDS stage
constexpr int kGroupM = 8;

// LDS ring discipline: the K slices are copied global -> LDS by the DMA path
// and the MFMA fragments read by inline-assembly ds_read_b128, with every wait
// placed by hand (the helpers in mx_device.h).

// Chunk swizzle of LDS row r: 16-byte chunk c is stored at c ^ swz(r).  A
// 16-lane phase of a fragment read (rows r0 .. r0 + 15, one logical chunk)
// then touches 16 distinct bank groups of 16 bytes: row r sits in group
// 4 (r % 4) + chunk of its 256 bytes, and swz takes all four values over
// r >> 2 for each r % 4.  (The same holds for 8-row phases over 32 banks.)
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 3) ^ ((r >> 3) & 1); }

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

// silu(g) = g / (1 + e^-g), the quotient through the reciprocal instruction
// (1 ulp) rather than the IEEE division sequence (about ten instructions per
// element in the epilogue): the result is rounded to bf16 anyway.  g -> -inf:
// 1 / inf = 0, so silu -> -0; g -> +inf: g.
__device__ __forceinline__ float silu(float g) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g));
}

// Fused QKV epilogue for one rotary pair: packed columns c and c + 32 (c in the
// low 32-column block of a 64-column group) of token row t, fp32 values lo,
// hi, with the token's KV slot and the pair's (cos, sin) already read.  q and k
// heads are rotated (rotate-half pairing, dims d_lo and d_lo + hd/2) and
// rounded once; q goes to q_out, k and v to their slots in the pools.
__device__ __forceinline__ void qkv_pair_store(uint16_t* __restrict__ q_out,
                                               uint16_t* __restrict__ k_pool,
                                               uint16_t* __restrict__ v_pool, int nq, int nkv,
                                               int hd, int t, int c, float lo, float hi,
                                               int64_t slot, float2 cs) {
  const int head = c / hd, within = c % hd;
  if (head < nq + nkv) {
    const int d_lo = 32 * (within / 64) + (within % 32);
    const float rlo = lo * cs.x - hi * cs.y;
    const float rhi = hi * cs.x + lo * cs.y;
    uint16_t* dst;
    int step;  // element distance from dim d_lo to dim d_lo + hd/2
    if (head < nq) {
      dst = q_out + ((int64_t)t * nq + head) * hd + d_lo;
      step = hd / 2;
    } else {
      // key pages blocked by 32 dims: [d / 32][16 slots][32]
      const int64_t page = slot / 16;
      dst = k_pool + (page * nkv + (head - nq)) * 16 * hd + (d_lo / 32) * 512 + (slot % 16) * 32 +
            d_lo % 32;
      step = 8 * hd;
    }
    dst[0] = f32_to_bf16(rlo);
    dst[step] = f32_to_bf16(rhi);
  } else {
    const int64_t page = slot / 16;
    uint16_t* dst = v_pool + ((page * nkv + (head - nq - nkv)) * hd) * 16 + slot % 16;
    dst[(int64_t)within * 16] = f32_to_bf16(lo);
    dst[(int64_t)(within + 32) * 16] = f32_to_bf16(hi);
  }
}

// The (cos, sin) of packed column c (any column of a 64-column group) of
// token t; in bounds for every c (v heads read a row of the table too).
__device__ __forceinline__ int rope_index(int t, int c, int hd) {
  const int within = c % hd;
  return t * (hd / 2) + 32 * (within / 64) + (within % 32);
}

// QKV epilogue of one wave's block (rows r0.., the 64 columns c0..: one
// 64-column group of one head, i.e. the two 32-column halves of its rotary
// pairs).  q and k heads are rotated and rounded once; q goes to q_out, k to
// its pool slot ([d / 32][16 slots][32] pages), v to the transposed value
// pages [page][kv head][dim][16 slots].  Per 32-row block the rounded values
// are staged in LDS, like the outputs of the other epilogues, and written in
// 16-byte runs: q and k read back token-major (8 consecutive dims of one
// token per run), v dim-major, 8 consecutive tokens of one dim per run
// wherever they fill 8 consecutive slots starting at a multiple of 8, in any
// position in the block (a chunk's start need not line up with the rows); the
// tokens left over are stored one value at a time.  Each block first issues
// its reads (this lane's token slot, the rotary cos/sin), so that no wait on
// them also waits for a store (one counter tracks both).
constexpr int kQkRow = 64 + 8;  // bf16 per staged token row (q, k)
constexpr int kVRow = 32 + 8;   // bf16 per staged dim row (v)
constexpr int kQkvStageHalves = 64 * kVRow > 32 * kQkRow ? 64 * kVRow : 32 * kQkRow;

__device__ __forceinline__ int64_t lane_slot(int64_t s, int l) {  // s of lane l (uniform l)
  const int lo = __builtin_amdgcn_readlane((int)(uint32_t)s, l);
  const int hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)s >> 32), l);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

template <int MA, int NQ>
__device__ __forceinline__ void qkv_epilogue(const f32x4 (&acc)[MA][NQ], int M, int N, int r0,
                                             int c0, int lane, const float2* __restrict__ rope_cs,
                                             const int64_t* __restrict__ tok_slot,
                                             uint16_t* __restrict__ q_out,
                                             uint16_t* __restrict__ k_pool,
                                             uint16_t* __restrict__ v_pool, int nq, int nkv,
                                             int hd, MX_LDS uint16_t* st) {
  static_assert(NQ == 4, "one 64-column group per wave");
  if (c0 >= N) return;  // (wave-uniform)
  // accumulator layout: block (a, j) holds rows 16 a + crow .. + 3 of column
  // 16 j + ccol in this lane
  const int ccol = lane & 15, crow = 4 * (lane >> 4);
  const int head = c0 / hd, within0 = c0 % hd;
  const bool is_v = head >= nq + nkv, is_q = head < nq;
  // dims of the low and high 32-column blocks (q / k: the packed rotary halves)
  const int d_lo = is_v ? within0 : 32 * (within0 / 64);
  const int d_hi = is_v ? within0 + 32 : d_lo + hd / 2;
#pragma unroll
  for (int i = 0; i < MA / 2; i++) {  // 32-row blocks: accumulator rows 2 i, 2 i + 1
    const int rb = r0 + i * 32;
    // 1. reads: the slot of token rb + lane % 32, the (cos, sin) of this lane's
    // elements (rows 16 h + crow + v, low columns 16 j + ccol, h, j < 2)
    const int64_t myslot = tok_slot[min(rb + (lane & 31), M - 1)];
    float2 cs[16];
    if (!is_v) {
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int h = e >> 3, j = (e >> 2) & 1, v = e & 3;
        const int row = min(rb + 16 * h + crow + v, M - 1);
        cs[e] = rope_cs[(int64_t)row * (hd / 2) + d_lo + 16 * j + ccol];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (!is_v) {
      // 2. rotate, round, stage token-major: [token][low 32 dims, high 32 dims]
      // (a pair's halves are columns c and c + 32: blocks j and j + 2, same lane)
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int h = e >> 3, j = (e >> 2) & 1, v = e & 3;
        const int t = 16 * h + crow + v, c = 16 * j + ccol;
        const float lo = acc[2 * i + h][j][v], hi = acc[2 * i + h][j + 2][v];
        st[t * kQkRow + c] = f32_to_bf16(lo * cs[e].x - hi * cs[e].y);
        st[t * kQkRow + 32 + c] = f32_to_bf16(hi * cs[e].x + lo * cs[e].y);
      }
      lgkm_wait<0>();  // (and no access below moves above the staging)
      // 3. read back token (lane / 8) + 8 q, dims 8 (lane % 8) .. + 7 of the 64
      u32x4 out[4];
#pragma unroll
      for (int q = 0; q < 4; q++)
        out[q] = *reinterpret_cast<const MX_LDS u32x4*>(st + ((lane >> 3) + 8 * q) * kQkRow +
                                                        8 * (lane & 7));
      lgkm_wait<0>();  // the block is read back before the next one is staged
      const int p = lane & 7;
      const int dim = (p < 4 ? d_lo : d_hi) + 8 * (p & 3);
#pragma unroll
      for (int q = 0; q < 4; q++) {
        const int t = (lane >> 3) + 8 * q;
        const int64_t slot = __shfl(myslot, t);  // (every lane takes part)
        if (rb + t >= M) continue;
        uint16_t* dst;
        if (is_q) {
          dst = q_out + ((int64_t)(rb + t) * nq + head) * hd + dim;
        } else {
          dst = k_pool + ((slot >> 4) * nkv + (head - nq)) * 16 * hd + (dim >> 5) * 512 +
                (slot & 15) * 32 + (dim & 31);
        }
        *reinterpret_cast<u32x4*>(dst) = out[q];
      }
    } else {
      // 2. stage dim-major: [dim (low 32, high 32)][token]; this lane's four
      // consecutive tokens of a block are one 8-byte write
#pragma unroll
      for (int h = 0; h < 2; h++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          const f32x4 a = acc[2 * i + h][j];
          u32x2 w;
          w[0] = pack_bf16x2(a[0], a[1]);
          w[1] = pack_bf16x2(a[2], a[3]);
          *reinterpret_cast<MX_LDS u32x2*>(st + (16 * j + ccol) * kVRow + 16 * h + crow) = w;
        }
      lgkm_wait<0>();
      // runs: token t starts one where its slot is a multiple of 8 and token
      // t + 7 holds the slot 7 further (then the eight tokens are consecutive
      // positions of one request: a page belongs to one request)
      const int tl = lane & 31;
      const int64_t s7 = __shfl(myslot, min(tl + 7, 31));
      const bool start = tl + 7 < 32 && rb + tl + 7 < M && (myslot & 7) == 0 && s7 == myslot + 7;
      uint32_t starts = (uint32_t)__ballot(start);
      const int nrow = min(32, M - rb);
      uint32_t single = nrow >= 32 ? ~0u : ((1u << nrow) - 1u);
      for (uint32_t m = starts; m; m &= m - 1) single &= ~(0xFFu << __builtin_ctz(m));
      const int vh = head - nq - nkv;
      const int dim = within0 + lane;  // lane l writes dim row l of the staging
      const MX_LDS uint16_t* srow = st + lane * kVRow;
      for (; starts; starts &= starts - 1) {
        const int t = __builtin_ctz(starts);
        const int64_t slot = lane_slot(myslot, t);
        u32x4 v;
        if ((t & 7) == 0) {
          v = *reinterpret_cast<const MX_LDS u32x4*>(srow + t);
        } else {
#pragma unroll
          for (int e = 0; e < 4; e++) v[e] = (uint32_t)srow[t + 2 * e] | ((uint32_t)srow[t + 2 * e + 1] << 16);
        }
        *reinterpret_cast<u32x4*>(v_pool + (((slot >> 4) * nkv + vh) * hd + dim) * 16 + (slot & 15)) = v;
      }
      for (; single; single &= single - 1) {
        const int t = __builtin_ctz(single);
        const int64_t slot = lane_slot(myslot, t);
        v_pool[(((slot >> 4) * nkv + vh) * hd + dim) * 16 + (slot & 15)] = srow[t];
      }
      lgkm_wait<0>();
    }
  }
}

// Output staging of the plain, residual and SwiGLU epilogues.  The
// matrix-core layout gives a lane one column of four rows per 32 x 32 block, so
// writing it out directly takes one 2-byte store (and one 2-byte residual load)
// per element: 64-128 store instructions per lane per tile, and a CU issues
// about one vector memory instruction per 16 cycles, so the epilogue of a
// 256 x 256 tile cost 5-15 us.  Instead each wave stages one 32-row block of
// its fp32 results at a time in LDS (the operand ring, free once the main loop
// is done) and reads it back as runs of 8 consecutive columns of one row: a
// lane then moves 8 outputs, and 8 residuals, per 16-byte access.  The sums
// and roundings are the same as unstaged.  Staged rows are padded by 4 floats
// so that the rows 4 apart, which one write instruction covers, fall on other
// banks.
constexpr int kStageRow = 64 + 4;              // floats per staged row (64 columns)
constexpr int kStageFloats = 32 * kStageRow;   // one wave's 32-row block
constexpr int kStageRowSw = 32 + 4;            // SwiGLU: 32 output columns per wave

// Plain or residual epilogue of one wave's block (rows r0.., columns c0..,
// 64 columns).  Every residual read (indices clamped into range) is issued
// first, then per 32-row block the staging, the sums rounded to bf16 and the
// stores.  Rows whose stride is not a multiple of 8 elements, and the columns
// at the N edge, take 2-byte accesses.  R must not overlap C.
template <int MA, int NQ, bool RESIDUAL>
__device__ __forceinline__ void store_epilogue(const f32x4 (&acc)[MA][NQ], int M, int N, int r0,
                                               int c0, int lane, const uint16_t* __restrict__ R,
                                               int ldr, uint16_t* __restrict__ C, int ldc,
                                               MX_LDS float* st) {
  static_assert(NQ == 4, "the staging holds 64 columns per wave");
  constexpr int MB = MA / 2;  // 32-row blocks
  const int ccol = lane & 15, crow = 4 * (lane >> 4);  // accumulator layout
  const int rq = lane >> 3, col = c0 + 8 * (lane & 7);  // read-back: rows rq + 8 q, 8 columns
  const bool vec = ldc % 8 == 0 && (!RESIDUAL || ldr % 8 == 0) && col + 8 <= N;
  u32x4 res[MB][4];
#pragma unroll
  for (int i = 0; i < MB; i++)
#pragma unroll
    for (int q = 0; q < 4; q++) {
      res[i][q] = u32x4{0, 0, 0, 0};
      if constexpr (RESIDUAL) {
        const uint16_t* rp = R + (int64_t)min(r0 + i * 32 + rq + 8 * q, M - 1) * ldr;
        if (vec) {
          res[i][q] = *reinterpret_cast<const u32x4*>(rp + col);
        } else {
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const uint32_t lo = rp[min(col + e, N - 1)], hi = rp[min(col + e + 1, N - 1)];
            res[i][q][e / 2] = lo | (hi << 16);
          }
        }
      }
    }
#pragma unroll
  for (int i = 0; i < MB; i++) {
#pragma unroll
    for (int h = 0; h < 2; h++)
#pragma unroll
      for (int v = 0; v < 4; v++)
#pragma unroll
        for (int j = 0; j < NQ; j++)
          st[(16 * h + crow + v) * kStageRow + 16 * j + ccol] = acc[2 * i + h][j][v];
    lgkm_wait<0>();  // (and no access below moves above the staging)
    u32x4 out[4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const MX_LDS f32x4* sp =
          reinterpret_cast<const MX_LDS f32x4*>(st + (rq + 8 * q) * kStageRow + 8 * (lane & 7));
      const f32x4 lo = sp[0], hi = sp[1];
#pragma unroll
      for (int e = 0; e < 2; e++) {
        out[q][e] = pack_bf16x2(lo[2 * e] + __uint_as_float(res[i][q][e] << 16),
                                lo[2 * e + 1] + __uint_as_float(res[i][q][e] & 0xFFFF0000u));
        out[q][2 + e] = pack_bf16x2(hi[2 * e] + __uint_as_float(res[i][q][2 + e] << 16),
                                    hi[2 * e + 1] + __uint_as_float(res[i][q][2 + e] & 0xFFFF0000u));
      }
    }
    lgkm_wait<0>();  // the block is read back before the next one is staged
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const int row = r0 + i * 32 + rq + 8 * q;
      if (row >= M || col >= N) continue;
      uint16_t* cp = C + (int64_t)row * ldc + col;
      if (vec) {
        *reinterpret_cast<u32x4*>(cp) = out[q];
      } else {
#pragma unroll
        for (int e = 0; e < 8; e++)
          if (col + e < N) cp[e] = (uint16_t)(out[q][e / 2] >> (16 * (e & 1)));
      }
    }
  }
}

// The fp32 partial sums of one K split, through the same staging: 8
// consecutive columns of one row per lane and run, two 16-byte stores (rows
// of N % 4 != 0 floats, and the columns at the N edge, take 4-byte stores).
template <int MA, int NQ>
__device__ __forceinline__ void split_epilogue(const f32x4 (&acc)[MA][NQ], int M, int N, int r0,
                                               int c0, int lane, float* __restrict__ P,
                                               MX_LDS float* st) {
  static_assert(NQ == 4, "the staging holds 64 columns per wave");
  const int ccol = lane & 15, crow = 4 * (lane >> 4);  // accumulator layout
  const int rq = lane >> 3, col = c0 + 8 * (lane & 7);
  const bool vec = N % 4 == 0 && col + 8 <= N;
#pragma unroll
  for (int i = 0; i < MA / 2; i++) {
#pragma unroll
    for (int h = 0; h < 2; h++)
#pragma unroll
      for (int v = 0; v < 4; v++)
#pragma unroll
        for (int j = 0; j < NQ; j++)
          st[(16 * h + crow + v) * kStageRow + 16 * j + ccol] = acc[2 * i + h][j][v];
    lgkm_wait<0>();
    f32x4 lo[4], hi[4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const MX_LDS f32x4* sp =
          reinterpret_cast<const MX_LDS f32x4*>(st + (rq + 8 * q) * kStageRow + 8 * (lane & 7));
      lo[q] = sp[0];
      hi[q] = sp[1];
    }
    lgkm_wait<0>();
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const int row = r0 + i * 32 + rq + 8 * q;
      if (row >= M || col >= N) continue;
      float* pp = P + (int64_t)row * N + col;
      if (vec) {
        reinterpret_cast<f32x4*>(pp)[0] = lo[q];
        reinterpret_cast<f32x4*>(pp)[1] = hi[q];
      } else {
#pragma unroll
        for (int e = 0; e < 8; e++)
          if (col + e < N) pp[e] = e < 4 ? lo[q][e] : hi[q][e - 4];
      }
    }
  }
}

// SwiGLU epilogue of one wave's block: packed columns c0.. hold 32-column
// blocks of gate and up of the same 32 features; the 32 outputs (columns
// c0 / 2 ..) go to C row-major or, c_tiled, in the projection-input tile
// layout, through the same staging as above (ldc a multiple of 32).
template <int MA, int NQ>
__device__ __forceinline__ void swiglu_epilogue(const f32x4 (&acc)[MA][NQ], int M, int N, int r0,
                                                int c0, int lane, uint16_t* __restrict__ C,
                                                int ldc, bool c_tiled, MX_LDS float* st) {
  static_assert(NQ == 4, "one gate/up pair per wave");
  // accumulator layout; gate column c pairs with up column c + 32 (blocks j, j + 2)
  const int ccol = lane & 15, crow = 4 * (lane >> 4);
  const int rq = lane >> 2, col = c0 / 2 + 8 * (lane & 3);  // read-back: rows rq + 16 q
  if (c0 >= N) return;  // (wave-uniform)
#pragma unroll
  for (int i = 0; i < MA / 2; i++) {
#pragma unroll
    for (int h = 0; h < 2; h++)
#pragma unroll
      for (int v = 0; v < 4; v++)
#pragma unroll
        for (int j = 0; j < 2; j++)
          st[(16 * h + crow + v) * kStageRowSw + 16 * j + ccol] =
              silu(acc[2 * i + h][j][v]) * acc[2 * i + h][j + 2][v];
    lgkm_wait<0>();
    u32x4 out[2];
#pragma unroll
    for (int q = 0; q < 2; q++) {
      const MX_LDS f32x4* sp =
          reinterpret_cast<const MX_LDS f32x4*>(st + (rq + 16 * q) * kStageRowSw + 8 * (lane & 3));
      const f32x4 lo = sp[0], hi = sp[1];
      out[q] = u32x4{pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]), pack_bf16x2(hi[0], hi[1]),
                     pack_bf16x2(hi[2], hi[3])};
    }
    lgkm_wait<0>();
#pragma unroll
    for (int q = 0; q < 2; q++) {
      const int row = r0 + i * 32 + rq + 16 * q;
      if (row >= M) continue;
      *reinterpret_cast<u32x4*>(C + (c_tiled ? tile_index(row, col, ldc) : (int64_t)row * ldc + col)) =
          out[q];
    }
  }
}

template <int BM, int BN, int WM, int WN, int NS, int EPI, bool SPLIT>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void gemm_kernel(GemmArgs a, int tiles_m,
                                                                           int tiles_n,
                                                                           int k_chunks) {
  constexpr int WAVES_N = BN / WN;
  constexpr int NWAVES = (BM / WM) * WAVES_N;
  // 16 x 16 output blocks of v_mfma_f32_16x16x32_bf16: MA rows of them per
  // wave, NQ columns; a slice (32 of K) is one product per block
  constexpr int MA = WM / 16, NQ = WN / 16, MH = MA / 2;
  constexpr int ROWB = BKS * 2;                // bytes of one tile row in a stage (64)
  constexpr int STAGE = (BM + BN) * ROWB;      // bytes per LDS stage
  constexpr int L = STAGE / 1024 / NWAVES;     // DMA instructions per wave per stage
  static_assert(L * NWAVES * 1024 == STAGE, "stage does not split into whole DMA rows");
  constexpr int VM_KEEP = (NS - 2) * L;        // in flight after the oldest stage landed
  constexpr int NR0 = NQ + MH;                 // fragment reads of phase 0 (B, first A half)
  constexpr int NR1 = MH;                      // fragment reads of phase 1 (second A half)
  static_assert(MA % 2 == 0 && NQ == 4, "two A halves; 64 columns per wave");
  static_assert(NR0 + NR1 <= 15, "lgkmcnt range");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const unsigned sbase = (unsigned)(size_t)(MX_LDS char*)smem;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wave_m = wave / WAVES_N, wave_n = wave % WAVES_N;
  int tm, tn;
  tile_coords(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kz = blockIdx.y;
  const int c_beg = kz * k_chunks / (int)gridDim.y, c_end = (kz + 1) * k_chunks / (int)gridDim.y;
  const int kbeg = c_beg * BK;
  const int nk = (c_end - c_beg) * (BK / BKS);

  // DMA: instruction j (wave w issues j = w L .. w L + L - 1) fills rows
  // 16 j .. 16 j + 15 of the stacked A|B tile; lane l lands at row 16 j + l / 4,
  // stored chunk l % 4, which holds logical chunk (l % 4) ^ swz(row).
  // (an instruction's 16 rows are all A or all B: BM is a multiple of 16, so
  // which operand an instruction reads is wave-uniform.)  Each lane keeps a
  // pointer to its 16 bytes of the next slice to issue, advanced by a scalar
  // step after every issue (no per-slice address multiply), and the LDS
  // destination is scalar arithmetic on the wave index.
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint16_t* dsrc[L];
  int64_t dstep[L];
  // A element (m, k) at A + (m / 16) a_blk + (m % 16) a_row + (k / 32) a_kstep
  // + k % 32: row-major (16 lda, lda, 32) or the activation tiles
  // (tile_row_pitch(lda), 32, 512), where the 16 rows of an instruction are one
  // contiguous kilobyte
  const int64_t a_blk = a.a_tiled ? tile_row_pitch(a.lda) : 16 * (int64_t)a.lda;
  const int a_row = a.a_tiled ? 32 : a.lda;
  const int a_kstep = a.a_tiled ? 512 : BKS;
#pragma unroll
  for (int i = 0; i < L; i++) {
    const int row0 = (wave_s * L + i) * 16;  // first tile row of instruction i
    const int row = row0 + (lane >> 2);
    const int c = (lane & 3) ^ swz(row);
    if (row0 < BM) {
      const int m = min(m0 + row, a.M - 1);
      dsrc[i] = a.A + (int64_t)(m >> 4) * a_blk + (int64_t)(m & 15) * a_row +
                (int64_t)(kbeg >> 5) * a_kstep + c * 8;
      dstep[i] = a_kstep;
    } else {
      const int n = min(n0 + row - BM, a.N - 1);
      dsrc[i] = a.B + (int64_t)(n >> 4) * a.b_blk + (int64_t)(n & 15) * a.b_row +
                (int64_t)(kbeg >> 5) * a.b_kstep + c * 8;
      dstep[i] = a.b_kstep;
    }
  }
  // DMA instruction i of slice st into its LDS slot; slices are issued in
  // order, and past the end the last slice is fetched again (never read)
  auto dma_one = [&](int i, int st) {
    const unsigned slot = sbase + (unsigned)((st % NS) * STAGE);
    dma16(dsrc[i], slot + (unsigned)((wave_s * L + i) * 1024));
    if (st < nk - 1) dsrc[i] += dstep[i];
  };

  f32x4 acc[MA][NQ];
#pragma unroll
  for (int i = 0; i < MA; i++)
#pragma unroll
    for (int j = 0; j < NQ; j++) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // A fragment of 16-row block a: lane l holds row 16 a + l % 16, logical
  // chunk l / 16 (8 of the slice's 32 K values); B likewise for its columns
  const int frow = lane & 15, fk = lane >> 4;
  unsigned aoff[MA], boff[NQ];
#pragma unroll
  for (int i = 0; i < MA; i++) {
    const int r = wave_m * WM + i * 16 + frow;
    aoff[i] = r * ROWB + (((unsigned)fk ^ swz(r)) << 4);
  }
#pragma unroll
  for (int j = 0; j < NQ; j++) {
    const int r = wave_n * WN + j * 16 + frow;
    boff[j] = (BM + r) * ROWB + (((unsigned)fk ^ swz(r)) << 4);
  }
  // A slice runs in two phases, the first and second half of the wave's A
  // blocks against all its B blocks: fa0 and fa1 hold the two halves, fb[p]
  // the B fragments of slices of parity p (the next slice's arrive while the
  // second phase still uses this one's).
  u32x4 fa0[MH], fa1[MH], fb[2][NQ];
  // phase-0 fragment r of slice st (B first, then the first A half), into fb[p]
  auto read0 = [&](int p, int st, int r) {
    const unsigned slot = sbase + (unsigned)((st % NS) * STAGE);
    if (r < NQ)
      fb[p][r] = lds_read16(slot + boff[r]);
    else
      fa0[r - NQ] = lds_read16(slot + aoff[r - NQ]);
  };
  // phase-1 fragment r of slice st (the second A half)
  auto read1 = [&](int st, int r) {
    const unsigned slot = sbase + (unsigned)((st % NS) * STAGE);
    fa1[r] = lds_read16(slot + aoff[MH + r]);
  };
  constexpr int NM = MH * NQ;  // MFMAs per phase
  auto mfma0 = [&](int p, int idx) {
    const int i = idx / NQ, j = idx % NQ;
    acc[i][j] = mfma16(as_bf16x8(fa0[i]), as_bf16x8(fb[p][j]), acc[i][j]);
  };
  auto mfma1 = [&](int p, int idx) {
    const int i = idx / NQ, j = idx % NQ;
    acc[MH + i][j] = mfma16(as_bf16x8(fa1[i]), as_bf16x8(fb[p][j]), acc[MH + i][j]);
  };

  // One slice (p = kt % 2, a constant at every call): its two phases.  The
  // MFMAs of each phase go out one at a time, with the slice's memory
  // instructions spread between them (the DMA of slice kt + NS - 1 among the
  // first phase's, the next slice's phase-0 fragment reads among the
  // second's), so that a wave keeps the matrix core fed while it issues them:
  // with the instructions in bursts, the two waves of a SIMD, lined up by the
  // barrier, issued theirs at the same time and the matrix core idled
  // meanwhile.  `more` issues the fragment reads of the next slice's first
  // phase.  The last slice must not: the compiler sees the result of a read
  // that is never consumed as dead and may hand its registers to the epilogue
  // while the read is still in flight, and the landing data would then
  // overwrite them.
  auto slice = [&](int kt, bool more, auto parity) {
    constexpr int p = decltype(parity)::value;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int r = 0; r < NR1; r++) read1(kt, r);
    lgkm_wait<NR1>();  // the phase-0 fragments (older reads) have landed
    pin(fa0);
    pin(fb[p]);
    // slot (kt + NS - 1) % NS was last read in slice kt - 1, before its barrier
#pragma unroll
    for (int idx = 0; idx < NM; idx++) {
      mfma0(p, idx);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < L; i++)
        if (i * NM / L == idx) dma_one(i, kt + NS - 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    // (every fragment buffer of a phase stays live across it, so that no
    // read's destination is a register an MFMA of the phase took as a source)
    pin(fa0);
    pin(fb[p]);
    // own DMA of stage kt + 1 landed, own reads of stage kt done; after the
    // barrier everyone's are, so stage kt + 1 is readable and slot kt % NS free
    vm_wait<VM_KEEP>();
    lgkm_wait<0>();
    pin(fa1);
    pin(fb[p]);
    wg_barrier();
#pragma unroll
    for (int idx = 0; idx < NM; idx++) {
      mfma1(p, idx);
      __builtin_amdgcn_sched_barrier(0);
      if (more) {
#pragma unroll
        for (int r = 0; r < NR0; r++)
          if (r * NM / NR0 == idx) read0(p ^ 1, kt + 1, r);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    pin(fa1);
    pin(fb[p]);
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;

#pragma unroll
  for (int st = 0; st < NS - 1; st++)
#pragma unroll
    for (int i = 0; i < L; i++) dma_one(i, st);
  vm_wait<VM_KEEP>();
  wg_barrier();
#pragma unroll
  for (int r = 0; r < NR0; r++) read0(0, 0, r);
  // nk is even (K is a multiple of 64), so slices pair up by parity
  for (int kt = 0; kt < nk - 2; kt += 2) {
    slice(kt, true, P0{});
    slice(kt + 1, true, P1{});
  }
  slice(nk - 2, true, P0{});
  slice(nk - 1, false, P1{});
  // drain: no DMA may still target this workgroup's LDS when it exits (no
  // fragment read is outstanding: the last slice waited for all of them)
  vm_wait<0>();

  // epilogue
  if constexpr (EPI == EPI_QKV && !SPLIT) {
    static_assert(NWAVES * kQkvStageHalves * 2 <= NS * STAGE, "the staging does not fit the ring");
    wg_barrier();  // every wave is done reading the ring
    MX_LDS uint16_t* st =
        reinterpret_cast<MX_LDS uint16_t*>((MX_LDS char*)smem) + wave_s * kQkvStageHalves;
    const QkvEpilogue& e = a.qkv;
    qkv_epilogue<MA, NQ>(acc, a.M, a.N, m0 + wave_m * WM, n0 + wave_n * WN, lane, e.rope_cs,
                         e.tok_slot, e.q_out, e.k_pool, e.v_pool, e.nq, e.nkv, e.head_dim, st);
    return;
  }
  if constexpr (!SPLIT && (EPI == EPI_STORE || EPI == EPI_RESIDUAL || EPI == EPI_SWIGLU)) {
    static_assert(NWAVES * kStageFloats * 4 <= NS * STAGE, "the staging does not fit the ring");
    wg_barrier();  // every wave is done reading the ring
    MX_LDS float* st = reinterpret_cast<MX_LDS float*>((MX_LDS char*)smem) + wave_s * kStageFloats;
    if constexpr (EPI == EPI_SWIGLU)
      swiglu_epilogue<MA, NQ>(acc, a.M, a.N, m0 + wave_m * WM, n0 + wave_n * WN, lane, a.C, a.ldc,
                              a.c_tiled != 0, st);
    else
      store_epilogue<MA, NQ, EPI == EPI_RESIDUAL>(acc, a.M, a.N, m0 + wave_m * WM,
                                                  n0 + wave_n * WN, lane, a.R, a.ldr, a.C, a.ldc,
                                                  st);
    return;
  }
  if constexpr (SPLIT) {  // this split's fp32 plane, [M][N]
    static_assert(NWAVES * kStageFloats * 4 <= NS * STAGE, "the staging does not fit the ring");
    wg_barrier();
    MX_LDS float* st = reinterpret_cast<MX_LDS float*>((MX_LDS char*)smem) + wave_s * kStageFloats;
    split_epilogue<MA, NQ>(acc, a.M, a.N, m0 + wave_m * WM, n0 + wave_n * WN, lane,
                           a.partial + (int64_t)kz * a.M * a.N, st);
  }
}

// Plain or residual reduce, four columns per thread (N, ldc and ldr multiples
// of 4): 16-byte partial loads, 8-byte residual loads and stores, and every
// load of a thread's iteration issued before its store.
template <bool RESIDUAL>
__global__ __launch_bounds__(256) void splitk_reduce4_kernel(GemmArgs a, int ksplit) {
  const int nq4 = a.N / 4;
  const int64_t total = (int64_t)a.M * nq4;
  const f32x4* part = reinterpret_cast<const f32x4*>(a.partial);
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int row = (int)(idx / nq4), col = (int)(idx % nq4) * 4;
    f32x4 v = part[idx];
    for (int z = 1; z < ksplit; z++) {
      const f32x4 pz = part[z * total + idx];
      v[0] += pz[0]; v[1] += pz[1]; v[2] += pz[2]; v[3] += pz[3];
    }
    if constexpr (RESIDUAL) {
      const u32x2 r = *reinterpret_cast<const u32x2*>(a.R + (int64_t)row * a.ldr + col);
      v[0] += __uint_as_float(r[0] << 16);
      v[1] += __uint_as_float(r[0] & 0xFFFF0000u);
      v[2] += __uint_as_float(r[1] << 16);
      v[3] += __uint_as_float(r[1] & 0xFFFF0000u);
    }
    u32x2 w;
    w[0] = pack_bf16x2(v[0], v[1]);
    w[1] = pack_bf16x2(v[2], v[3]);
    *reinterpret_cast<u32x2*>(a.C + (int64_t)row * a.ldc + col) = w;
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
      const QkvEpilogue& e = a.qkv;
      qkv_pair_store(e.q_out, e.k_pool, e.v_pool, e.nq, e.nkv, e.head_dim, row, c, lo, hv,
                     e.tok_slot[row], e.rope_cs[rope_index(row, c, e.head_dim)]);
    } else if constexpr (EPI == EPI_SWIGLU) {
      const int fb = col / 32, w = col % 32;
      const int64_t gi = (int64_t)row * a.N + fb * 64 + w, ui = gi + 32;
      float g = 0.f, u = 0.f;
      for (int z = 0; z < ksplit; z++) {
        g += a.partial[z * plane + gi];
        u += a.partial[z * plane + ui];
      }
      a.C[a.c_tiled ? tile_index(row, col, a.ldc) : (int64_t)row * a.ldc + col] =
          f32_to_bf16(silu(g) * u);
    } else {
      const int64_t pi = (int64_t)row * a.N + col;
      float v = 0.f;
      for (int z = 0; z < ksplit; z++) v += a.partial[z * plane + pi];
      if constexpr (EPI == EPI_RESIDUAL) v += bf16_to_f32(a.R[(int64_t)row * a.ldr + col]);
      a.C[(int64_t)row * a.ldc + col] = f32_to_bf16(v);
    }
  }
}

struct Shape {
  int BM, BN;
  // time of one round of tile-units on the chip: a + b * (K slice length),
  // microseconds (least-squares fit over measured layer-shape GEMMs, all tile
  // shapes and K splits; the main loop is bound by its global->LDS feed, so a
  // unit's time grows with the bytes it streams)
  double a_us, b_us_per_k;
  int per_cu;       // tile-units one round holds per CU
  double feed_gbs;  // bytes a CU streams per microsecond (x1e3) with cold weights
};
// 256x256 and 128x256 run eight waves (2 per SIMD), the smaller shapes four.
// The last shape is 128x256 with a three-stage ring (72 KB of LDS), meant for
// two workgroups per CU; with the 16 x 16 x 32 main loop a 128x256 wave needs
// more than the 128 registers that four waves per SIMD leave, so it runs one
// per CU, and its figures (a fourth stage missing against the 128x256 shape)
// keep the model from choosing it.
constexpr Shape kShapes[] = {{256, 256, 3.471, 0.02443, 1, 33.8},
                             {128, 256, 0.978, 0.01544, 1, 42.1},
                             {128, 128, 0.615, 0.0115, 1, 43.3},
                             {64, 128, 0.0, 0.00729, 1, 49.6},
                             {128, 256, 0.978, 0.0287, 1, 42.1}};
constexpr int kNumShapes = 5;
constexpr int kFeedMaxM = 256;  // rows up to which the feed estimate is used
constexpr double kCUs = 256.0;

// Estimated time (us) of one GEMM launch with tile shape c and K split ks, in
// two regimes, or a negative value when the choice is not allowed.  Few rows
// (M <= kFeedMaxM): the layer's weights arrive cold from HBM and the busiest
// CU's feed bounds the time: its tile-units (ceil(units / 256)) times the
// bytes one unit streams (its A and B rows over its K slice) at the shape's
// per-CU fetch rate, plus a fixed cost.  More rows: the busiest CU runs
// ceil(units / (256 per_cu)) rounds of tile-units, and nothing beats
// streaming the operands from HBM once.  A K split adds the fp32 partial round
// trip and the reduce launch.  (Both fitted on cold timings of the layer GEMMs
// of the four layer shapes at their decode-only and mixed token counts, every
// tile shape and K split of 1, 2, 4 or 8: the picks are within 0.1-0.2% of the
// best measured in total and within 1% on the decode sizes, where the
// round-based estimate alone was 1.7-2.4% above the best.)  Every split from 1
// to 8 is a candidate: where the model moves to a split of 3, 5 or 6, the
// measured time fell on 10 of 11 such problems (7B down projection at 576 rows
// 92.8 -> 74.6 us with 128 x 256 tiles split three ways; Llama-3-8B down at
// 2304 rows 343.7 -> 304.7 us) and rose by 0.9% on the eleventh.
double estimate(int c, int ks, int M, int N, int K) {
  const double hbm = 5.0e12;
  if ((K / BK) / ks < 4) return -1.0;  // every split at least four 64-wide K chunks
  if (ks > 1 && (double)ks * M * N > (double)kMaxSplitFloats) return -1.0;
  const int BM = kShapes[c].BM, BN = kShapes[c].BN;
  const double tiles = (double)((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const double split_mb = ((double)ks * M * N * 8.0 + 2.0 * M * N) / 1e6;
  const double k_unit = (double)((K / BK + ks - 1) / ks * BK);  // the longest split
  if (M <= kFeedMaxM) {
    const double per_cu = std::ceil(tiles * ks / kCUs);
    const double unit_bytes = (double)(BN + std::min(BM, M)) * k_unit * 2.0;
    return per_cu * unit_bytes / (kShapes[c].feed_gbs * 1e3) + 12.06 +
           (ks > 1 ? 0.157 * split_mb + 0.15 : 0.0);
  }
  const double rounds = std::ceil(tiles * ks / (kCUs * kShapes[c].per_cu));
  const double t_units = rounds * (kShapes[c].a_us + kShapes[c].b_us_per_k * k_unit);
  const double t_mem = 2.0 * ((double)N * K + (double)M * K) / hbm * 1e6;
  return std::max(t_units, t_mem) + (ks > 1 ? 0.197 * split_mb + 3.39 : 0.0);
}

struct Pick {
  int cfg, ksplit;
  double t;
};

// The best (tile shape, K split) of one launch over all M rows.
Pick choose_one(int M, int N, int K) {
  Pick best{kNumShapes - 1, 1, 1e30};
  for (int c = 0; c < kNumShapes; c++)
    for (int ks = 1; ks <= 8; ks++) {
      const double t = estimate(c, ks, M, N, K);
      if (t < 0.0) break;
      if (t < best.t * 0.98) best = {c, ks, t};
    }
  return best;
}

// Launch plan of one GEMM.  Rows [0, m_main) run with tile shape cfg and K
// split ksplit; when m_main < M, the remaining rows run as a second GEMM of
// their own (tile shape tail_cfg, K split tail_ksplit) after the first.  The
// row split removes the last, mostly empty round of a problem whose tiles
// fill a few rounds and a little more (70B-shaped down projection at 8448
// rows: 1056 tiles of 256 x 256, 4.125 rounds of 256 CUs, run as 1024 tiles in
// four full rounds plus 256 rows split eight ways over K).
struct Plan {
  int cfg, ksplit;
  int m_main;
  int tail_cfg, tail_ksplit;
};

Plan plan_uncached(int M, int N, int K) {
  const Pick whole = choose_one(M, N, K);
  Plan best{whole.cfg, whole.ksplit, M, -1, 0};
  if (M <= 2 * kFeedMaxM) return best;
  double best_t = whole.t;
  // first part: whole rounds of one tile shape without a K split; second part:
  // the remaining rows, planned as a launch of their own (plus a launch gap)
  for (int c = 0; c < kNumShapes; c++) {
    const int BM = kShapes[c].BM, BN = kShapes[c].BN;
    const double slots = kCUs * kShapes[c].per_cu;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
    for (int j = tiles_m - 1; j >= 1 && M - j * BM <= 4 * kFeedMaxM; j--) {
      const double tiles = (double)j * tiles_n;
      const double frac = tiles / slots - std::floor(tiles / slots);
      if (frac > 0.0 && frac < 0.75) continue;  // only (nearly) full last rounds
      const double t_main = estimate(c, 1, j * BM, N, K);
      if (t_main < 0.0) continue;
      const Pick tail = choose_one(M - j * BM, N, K);
      const double t = t_main + tail.t + 4.0;
      if (t < best_t * 0.97) {
        best_t = t;
        best = {c, 1, j * BM, tail.cfg, tail.ksplit};
      }
    }
  }
  return best;
}

// Plans are cached per problem: the layer step plans four GEMMs per call.
Plan plan_gemm(int M, int N, int K) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, int>, Plan> cache;
  const auto key = std::make_tuple(M, N, K);
  {
    std::lock_guard<std::mutex> g(mu);
    auto it = cache.find(key);
    if (it != cache.end()) return it->second;
  }
  const Plan p = plan_uncached(M, N, K);
  std::lock_guard<std::mutex> g(mu);
  if (cache.size() > 4096) cache.clear();
  cache[key] = p;
  return p;
}

// Scratch (fp32 elements) that a plan's K split needs.
size_t plan_scratch(const Plan& p, int M, int N) {
  if (p.m_main < M) return p.tail_ksplit > 1 ? (size_t)p.tail_ksplit * (M - p.m_main) * N : 0;
  return p.ksplit > 1 ? (size_t)p.ksplit * M * N : 0;
}

// The GEMM of rows [m0, M) of a: every row-indexed operand moves by m0 rows
// (A, C, R and, for the QKV epilogue, the rotary table, the token slots and
// q_out; the pools are addressed through the slots).  In the tile layout row
// m0 starts a tile row only when m0 % 16 == 0, which the callers ensure.
GemmArgs rows_from(const GemmArgs& a, int m0) {
  GemmArgs t = a;
  t.M = a.M - m0;
  t.A = a.A + (a.a_tiled ? (int64_t)(m0 / 16) * tile_row_pitch(a.lda) : (int64_t)m0 * a.lda);
  if (t.C)
    t.C = a.C + (a.c_tiled ? (int64_t)(m0 / 16) * tile_row_pitch(a.ldc) : (int64_t)m0 * a.ldc);
  if (t.R) t.R = a.R + (int64_t)m0 * a.ldr;
  if (a.epilogue == EPI_QKV) {
    t.qkv.rope_cs = a.qkv.rope_cs + (int64_t)m0 * (a.qkv.head_dim / 2);
    t.qkv.tok_slot = a.qkv.tok_slot + m0;
    t.qkv.q_out = a.qkv.q_out + (int64_t)m0 * a.qkv.nq * a.qkv.head_dim;
  }
  return t;
}

template <int BM, int BN, int WM, int WN, int NS, int EPI, bool SPLIT>
hipError_t run(const GemmArgs& a, int ksplit, hipStream_t stream) {
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  const int threads = (BM / WM) * (BN / WN) * 64;
  const size_t lds = (size_t)NS * (BM + BN) * BKS * 2;
  dim3 grid(tiles_m * tiles_n, ksplit);
  gemm_kernel<BM, BN, WM, WN, NS, EPI, SPLIT><<<grid, threads, lds, stream>>>(a, tiles_m, tiles_n,
                                                                          a.K / BK);
  return hipGetLastError();
}

// reduce = false: a K split leaves its fp32 planes at a.partial for the caller
// to reduce.
template <int BM, int BN, int WM, int WN, int NS>
hipError_t run_shape(const GemmArgs& a, int ksplit, bool reduce, hipStream_t stream) {
  if (ksplit > 1) {
    hipError_t e = run<BM, BN, WM, WN, NS, EPI_STORE, true>(a, ksplit, stream);
    if (e != hipSuccess || !reduce) return e;
    const bool paired = a.epilogue == EPI_SWIGLU || a.epilogue == EPI_QKV;
    const int64_t total = (int64_t)a.M * (paired ? a.N / 2 : a.N);
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
    const bool by4 = !paired && a.N % 4 == 0 && a.ldc % 4 == 0 &&
                     (a.epilogue != EPI_RESIDUAL || a.ldr % 4 == 0);
    if (by4) {
      const int blocks4 = (int)std::min<int64_t>((total / 4 + 255) / 256, 4096);
      if (a.epilogue == EPI_RESIDUAL)
        splitk_reduce4_kernel<true><<<blocks4, 256, 0, stream>>>(a, ksplit);
      else
        splitk_reduce4_kernel<false><<<blocks4, 256, 0, stream>>>(a, ksplit);
      return hipGetLastError();
    }
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
    case EPI_QKV: return run<BM, BN, WM, WN, NS, EPI_QKV, false>(a, 1, stream);
    case EPI_SWIGLU: return run<BM, BN, WM, WN, NS, EPI_SWIGLU, false>(a, 1, stream);
    case EPI_RESIDUAL: return run<BM, BN, WM, WN, NS, EPI_RESIDUAL, false>(a, 1, stream);
    default: return run<BM, BN, WM, WN, NS, EPI_STORE, false>(a, 1, stream);
  }
}

template <int BM, int BN, int WM, int WN, int NS>
hipError_t set_lds_attr() {
  const int lds = NS * (BM + BN) * BKS * 2;
  hipError_t e;
#define MX_SET(EPI, SPLIT)                                                                  \
  e = hipFuncSetAttribute((const void*)gemm_kernel<BM, BN, WM, WN, NS, EPI, SPLIT>,             \
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
  hipError_t e = set_lds_attr<256, 256, 128, 64, 4>();
  if (e != hipSuccess) return e;
  e = set_lds_attr<128, 256, 64, 64, 4>();
  if (e != hipSuccess) return e;
  e = set_lds_attr<128, 128, 64, 64, 4>();
  if (e != hipSuccess) return e;
  e = set_lds_attr<64, 128, 32, 64, 4>();
  if (e != hipSuccess) return e;
  return set_lds_attr<128, 256, 64, 64, 3>();
}

size_t gemm_scratch_floats(int M, int N, int K) {
  return plan_scratch(plan_gemm(M, N, K), M, N);
}

void gemm_plan(int M, int N, int K, int out[5]) {
  const Plan p = plan_gemm(M, N, K);
  out[0] = p.cfg;
  out[1] = p.ksplit;
  out[2] = p.m_main;
  out[3] = p.tail_cfg;
  out[4] = p.tail_ksplit;
}

hipError_t launch_gemm(const GemmArgs& a, size_t ws_floats, hipStream_t stream) {
  return launch_gemm_config(a, ws_floats, -1, 0, stream);
}

int gemm_num_configs() { return kNumShapes; }

namespace {
hipError_t launch_shape(const GemmArgs& a, int cfg, int ksplit, bool reduce, hipStream_t stream) {
  switch (cfg) {
    case 0: return run_shape<256, 256, 128, 64, 4>(a, ksplit, reduce, stream);
    case 1: return run_shape<128, 256, 64, 64, 4>(a, ksplit, reduce, stream);
    case 2: return run_shape<128, 128, 64, 64, 4>(a, ksplit, reduce, stream);
    case 3: return run_shape<64, 128, 32, 64, 4>(a, ksplit, reduce, stream);
    default: return run_shape<128, 256, 64, 64, 3>(a, ksplit, reduce, stream);
  }
}

// A plan whose K split needs more scratch than there is runs that part unsplit.
Plan fit_scratch(Plan p, int M, int N, size_t ws_floats) {
  if (plan_scratch(p, M, N) > ws_floats) {
    if (p.m_main < M)
      p.tail_ksplit = 1;
    else
      p.ksplit = 1;
  }
  return p;
}

// reduce = false: the K split of the last part (the tail rows, or all rows
// without a row split) leaves its fp32 planes at a.partial for the caller.
hipError_t launch_plan(const GemmArgs& a, const Plan& p, bool reduce, hipStream_t stream) {
  if (p.m_main >= a.M) return launch_shape(a, p.cfg, p.ksplit, reduce, stream);
  GemmArgs head = a;
  head.M = p.m_main;
  hipError_t e = launch_shape(head, p.cfg, p.ksplit, true, stream);
  if (e != hipSuccess) return e;
  return launch_shape(rows_from(a, p.m_main), p.tail_cfg, p.tail_ksplit, reduce, stream);
}
}  // namespace

hipError_t launch_gemm_config(const GemmArgs& a, size_t ws_floats, int cfg, int ksplit,
                              hipStream_t stream) {
  if (a.M == 0) return hipSuccess;
  Plan p = plan_gemm(a.M, a.N, a.K);
  if (cfg >= 0 && cfg < kNumShapes) {
    p = Plan{cfg, ksplit >= 1 ? ksplit : 1, a.M, -1, 0};
    if (a.K / BK < p.ksplit) return hipErrorInvalidValue;
  }
  return launch_plan(a, fit_scratch(p, a.M, a.N, ws_floats), true, stream);
}

hipError_t launch_gemm_rows(const GemmArgs& a, size_t ws_floats, int m_main, int cfg,
                            int tail_cfg, int tail_ksplit, hipStream_t stream) {
  if (a.M == 0) return hipSuccess;
  if (m_main < 1 || m_main >= a.M || cfg < 0 || cfg >= kNumShapes || tail_cfg < 0 ||
      tail_cfg >= kNumShapes || tail_ksplit < 1 || a.K / BK < tail_ksplit)
    return hipErrorInvalidValue;
  if ((a.a_tiled || a.c_tiled) && m_main % 16) return hipErrorInvalidValue;
  const Plan p{cfg, 1, m_main, tail_cfg, tail_ksplit};
  if (plan_scratch(p, a.M, a.N) > ws_floats) return hipErrorInvalidValue;
  return launch_plan(a, p, true, stream);
}

hipError_t launch_gemm_unreduced(const GemmArgs& a, size_t ws_floats, int* split_row, int* ksplit,
                                 hipStream_t stream) {
  *split_row = a.M;
  *ksplit = 1;
  if (a.M == 0) return hipSuccess;
  const Plan p = fit_scratch(plan_gemm(a.M, a.N, a.K), a.M, a.N, ws_floats);
  const int ks = p.m_main < a.M ? p.tail_ksplit : p.ksplit;
  if (ks > 1) {
    *split_row = p.m_main < a.M ? p.m_main : 0;
    *ksplit = ks;
  }
  return launch_plan(a, p, false, stream);
}

}  // namespace mx
