// mx_kernels.h -- launchers of the gfx950 kernels (internal to libmx).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mx_device.h"

namespace mx {

struct AttnParams {
  const uint16_t* q;
  int64_t q_tok_stride;    // elements between consecutive tokens of q
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  uint16_t* out;
  int64_t out_tok_stride;  // elements between consecutive tokens of out (nq * head_dim)
  int32_t out_tiled;       // out in the tile layout (tile_index) instead of [T][nq][head_dim]
  const ReqDev* reqs;
  const int32_t* pages;
  const AttnItem* items;
  float* part_o;           // [parts][head_dim] unnormalised split outputs
  float* part_ml;          // [parts][2] running max (log2 units) and sum
  int32_t nq, nkv, group, split_pages;
  float scale_log2;        // softmax scale * log2(e)
  int32_t decode_only;     // no prefill items: decode keys and values are read non-temporally
};

hipError_t launch_paged_attn(const AttnParams& p, int n_items, const MergeItem* merges,
                             int n_merges, int head_dim, hipStream_t stream);

// Copies `bytes` (a multiple of 16, both ends 16-byte aligned) from pinned host
// memory, given by its device mapping, into device memory.  A kernel on the
// caller's stream rather than a copy-engine transfer, so that the first kernel
// of the step does not wait on a cross-engine signal.
hipError_t launch_upload(const void* host_mapped, void* dst, size_t bytes, hipStream_t stream);

// Plan kernel: tok_req/tok_pos/tok_slot of every new token from the request
// table and, when rope_cs is given, the RoPE (cos, sin) table [T][d/2] of the
// tokens' positions (angle formed and reduced in double precision).
hipError_t launch_token_map(const ReqDev* reqs, int R, int T, const int32_t* pages,
                            int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot,
                            const double* inv_freq, float2* rope_cs, int half,
                            hipStream_t stream);

// The token map with its rotary table and the first RMSNorm (below) in one
// launch: the first kernel of a layer step.
hipError_t launch_prologue(const ReqDev* reqs, int R, int T, const int32_t* pages,
                           int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot,
                           const double* inv_freq, float2* rope_cs, int half,
                           const uint16_t* x, const uint16_t* g, uint16_t* out, int H, float eps,
                           hipStream_t stream);

// RMSNorm: out[t] = x[t] / sqrt(mean(x[t]^2) + eps) * g, bf16 in/out, fp32 math.
// x is row-major [T][H]; out, a projection's input, is in the tile layout
// (tile_index, tile_elems(T, H) elements), H % 32 == 0.  The same holds for the
// RMSNorm outputs of the two launches around it.
hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* g, uint16_t* out, int T, int H,
                          float eps, hipStream_t stream);

// The residual split-K reduce fused with the RMSNorm of its result:
// x1 = bf16(sum_z partial[z] + R) over [M][H] fp32 planes (R, x1 [M][H] bf16),
// then h = RMSNorm(x1, g) (h in the tile layout).  One row per block of
// kNormThreads threads, each holding kNormChunks 16-byte chunks of the row in
// registers, so H % 32 == 0 and
// H <= kFusedNormMaxH; the first kNormPlanes planes are loaded ahead of the
// first sum, any further ones are summed as they arrive.
constexpr int kNormThreads = 512;
constexpr int kNormChunks = 2;
constexpr int kNormPlanes = 8;
constexpr int kFusedNormMaxH = 8 * kNormChunks * kNormThreads;
// Rows below split_row are complete already (x1 written): they are only
// normalised; the planes hold rows split_row .. M - 1, [ksplit][M - split_row][H].
hipError_t launch_reduce_residual_rmsnorm(const float* partial, int ksplit, const uint16_t* R,
                                          uint16_t* x1, const uint16_t* g, uint16_t* h, int M,
                                          int H, float eps, int split_row, hipStream_t stream);

// KV append of given k/v rows [T][nkv][d] into the pools.
hipError_t launch_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                            uint16_t* v_pool, const int64_t* tok_slot, int T, int nkv, int d,
                            hipStream_t stream);

// Gather of one request's keys/values (positions 0 .. len-1) into [len][nkv][d].
hipError_t launch_gather(const uint16_t* k_pool, const uint16_t* v_pool, const int32_t* pages,
                         int len, int nkv, int d, uint16_t* k_out, uint16_t* v_out,
                         hipStream_t stream);

// GEMM  C[M][N] = A[M][K] * B[N][K]^T, bf16 in, fp32 accumulate, fused epilogue.
enum GemmEpilogue : int {
  EPI_STORE = 0,    // C = acc
  EPI_RESIDUAL = 1, // C = acc + R   (R [M][N] bf16)
  EPI_SWIGLU = 2,   // B rows interleaved gate/up in 32-row blocks; C [M][N/2] = silu(gate) * up
  EPI_QKV = 3,      // QKV projection: RoPE on q/k heads, q -> q_out, k/v -> the paged pools
};

// Extra operands of the fused QKV epilogue.  The B rows of every q and k head
// (head_dim 128) are packed so that packed columns 64 g + w and 64 g + 32 + w
// of the head hold dims 32 g + w and 64 + 32 g + w: the two halves of a RoPE
// pair land in the same lane of two adjacent 32-column MFMA blocks.
struct QkvEpilogue {
  const float2* rope_cs;   // [T][head_dim / 2] (cos, sin)
  const int64_t* tok_slot; // [T] KV slot of each token
  uint16_t* q_out;         // [T][nq][head_dim]
  uint16_t* k_pool;        // [pages][nkv][head_dim / 32][16][32]
  uint16_t* v_pool;        // [pages][nkv][head_dim][16]
  int nq, nkv, head_dim;
};

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  const uint16_t* R;
  float* partial;      // split-K scratch [ksplit][M][N] fp32
  int M, N, K;
  int lda, ldb, ldc, ldr;
  int epilogue;
  QkvEpilogue qkv;
  // B element (n, k) sits at B + (n / 16) b_blk + (n % 16) b_row + (k / 32) b_kstep
  // + k % 32: row-major B is (16 ldb, ldb, 32) (set_b_row_major), the packed
  // weights are 16 x 32 tiles of 1 KB, [N / 16][K / 32][16][32] (set_b_tiled),
  // so that each DMA instruction reads one contiguous kilobyte
  int64_t b_blk, b_kstep;
  int b_row;
  // a_tiled: A in the activation tile layout (tile_index, K = lda) instead of
  // row-major; c_tiled: the SwiGLU output likewise (K = ldc).  Zero (the
  // default of an aggregate initialisation) is row-major.
  int a_tiled, c_tiled;
};

inline void set_b_row_major(GemmArgs& g) {
  g.b_blk = 16 * (int64_t)g.ldb;
  g.b_row = g.ldb;
  g.b_kstep = 32;
}
inline void set_b_tiled(GemmArgs& g) {
  g.b_blk = 16 * (int64_t)g.K;
  g.b_row = 32;
  g.b_kstep = 512;
}

// Chooses a tile shape and split for the problem; ws_floats is the fp32
// scratch available at args.partial.  A K split never needs more than
// kMaxSplitFloats of scratch (256 MB: enough for a three-way split of the
// down projection at a few thousand rows, where it saves 10-20%).
constexpr size_t kMaxSplitFloats = size_t(64) << 20;
hipError_t launch_gemm(const GemmArgs& args, size_t ws_floats, hipStream_t stream);
// The same with a forced tile shape (index < gemm_num_configs()) and K split;
// cfg < 0 uses the cost model.
hipError_t launch_gemm_config(const GemmArgs& args, size_t ws_floats, int cfg, int ksplit,
                              hipStream_t stream);
// A forced row split: rows [0, m_main) with tile shape cfg (no K split), then
// rows [m_main, M) as a GEMM of their own with tile_cfg and tail_ksplit.
hipError_t launch_gemm_rows(const GemmArgs& args, size_t ws_floats, int m_main, int cfg,
                            int tail_cfg, int tail_ksplit, hipStream_t stream);
// The cost model's plan without the last split-K reduce.  On return, rows
// [0, *split_row) are complete (epilogue applied); when *ksplit > 1, rows
// [*split_row, M) are left as fp32 planes at args.partial,
// [*ksplit][M - *split_row][N], without the epilogue (*split_row = M and
// *ksplit = 1 when every row is complete).
hipError_t launch_gemm_unreduced(const GemmArgs& args, size_t ws_floats, int* split_row,
                                 int* ksplit, hipStream_t stream);
int gemm_num_configs();
size_t gemm_scratch_floats(int M, int N, int K);
// The cost model's plan of an M x N x K problem: out[0] tile shape and out[1]
// K split of rows [0, out[2]); out[3] tile shape and out[4] K split of the
// remaining rows (out[2] == M: no row split, out[3] = -1).
void gemm_plan(int M, int N, int K, int out[5]);
hipError_t gemm_init();

// Weight packing: copies a [N][K] bf16 matrix into the GEMMs' tiled layout
// [N / 16][K / 32][16][32] (N % 16 == 0, K % 32 == 0), taking packed row n
// from source row perm(n): kind 0 identity, 1 the RoPE pair layout of the
// q/k rows of w_qkv, 2 the gate/up interleave.
hipError_t launch_pack_tiled(const uint16_t* src, uint16_t* dst, int N, int K, int kind, int nq,
                             int nkv, int d, int F, hipStream_t stream);

}  // namespace mx
