/*
 * mx.h -- C ABI of the MI355X (gfx950) multiplexed decoder-layer iteration.
 *
 * The problem statement this interface follows: a multiplexing worker runs
 * iterations whose batch mixes requests in the prefill phase (a chunk of
 * prompt tokens, possibly continuing an earlier chunk) with requests in the
 * decode phase (one new token each); prefill chunks are piggybacked onto the
 * running decode batch (paper Section 4.3, "Multiplexing Toggle"; Section 5.1,
 * chunked prefill with one chunk per iteration).  The engine keeps keys and
 * values in a paged cache (Section 5.1: the vLLM-based engine).  Every request
 * is described by its phase, its new-token count, the number of tokens already
 * cached and its page table.
 *
 * Conventions
 *  - All tensor pointers are DEVICE pointers unless marked [host].
 *  - bf16 tensors are passed as raw uint16 bit patterns.
 *  - Tokens of the batch are concatenated in request order; request r owns the
 *    n_new[r] consecutive rows starting at sum_{s<r} n_new[s].  Its i-th new
 *    token sits at position ctx_len + i and attends causally to the request's
 *    keys at positions 0 .. ctx_len + i.
 *  - Page size is 16 tokens.  The KV slot of position p of a request is
 *    pages[p / 16] * 16 + p % 16.
 *  - Pools (one for keys, one for values), per layer, bf16:
 *      k_pool[pool_pages][n_kv_heads][head_dim / 32][16][32]
 *                                                    (each page blocked by 32
 *                                                     dims: element (slot s,
 *                                                     dim e) of a page at
 *                                                     (e / 32) * 512 + s * 32
 *                                                     + e % 32, so that four
 *                                                     consecutive slots of a
 *                                                     32-dim block are one
 *                                                     contiguous 256-byte run)
 *      v_pool[pool_pages][n_kv_heads][head_dim][16]   (each page stored transposed,
 *                                                     so that the matrix-core
 *                                                     operands load contiguously)
 *    Byte offsets are 64-bit; pools larger than 4 GiB are supported.
 *  - Every device tensor and the workspace must be 16-byte aligned (the
 *    kernels move data in 16-byte vectors); a misaligned pointer is rejected
 *    with MX_ERR_INVALID.
 *  - Ownership: the caller allocates and owns every device buffer (weights,
 *    pools, activations, workspace) and the stream.  The library keeps no
 *    pointer after a call returns except for work already enqueued (a later
 *    call may record a completion event on the null stream for earlier calls
 *    made on it; never on another stream).  Host
 *    arrays (the batch) are read during the call only.  The library allocates
 *    nothing per call; on its first call on a device it allocates a small ring
 *    of pinned host staging buffers (grown, rarely, if a batch needs more) that
 *    lives until the process ends.
 *  - Errors: every input check runs on the host before anything is enqueued.
 *    On error nothing is enqueued, a status is returned and mx_last_error()
 *    (thread-local) gives a message.  No C++ exception crosses the ABI.  HIP
 *    launch errors map to MX_ERR_HIP; asynchronous faults surface at the
 *    caller's next synchronisation.
 *  - Threading: calls may come from several threads; calls that share one
 *    workspace must be ordered (same stream, or caller-side synchronisation).
 */
#ifndef MX_H
#define MX_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MX_OK = 0,
  MX_ERR_INVALID = 1,     /* malformed batch or shape, or a misaligned pointer */
  MX_ERR_NO_SPACE = 2,    /* a page table is too short for the request's positions */
  MX_ERR_TOO_LARGE = 3,   /* the workspace is too small for this batch */
  MX_ERR_UNSUPPORTED = 4, /* head_dim not in {64, 128}, page size not 16, ... */
  MX_ERR_NULL = 5,        /* a required pointer is NULL */
  MX_ERR_HIP = 6          /* a HIP runtime call failed */
} mx_status;

typedef enum { MX_PREFILL = 0, MX_DECODE = 1 } mx_phase;

/* One request of the iteration (the fields a scheduler hands to a worker). */
typedef struct {
  int32_t phase;        /* mx_phase */
  int32_t n_new;        /* new tokens this iteration: >= 1; exactly 1 for a decode */
  int32_t ctx_len;      /* tokens already cached before this iteration (>= 1 for a decode) */
  int32_t n_pages;      /* entries in pages[]: >= ceil((ctx_len + n_new) / 16) */
  const int32_t* pages; /* [host] page ids in [0, pool_pages) */
} mx_request;

typedef struct {
  int32_t num_reqs;       /* R >= 0; R == 0 is a no-op */
  const mx_request* reqs; /* [host] R requests */
} mx_batch;

typedef struct {
  int32_t n_q_heads, n_kv_heads; /* n_q_heads % n_kv_heads == 0; q head h reads kv head h / (n_q_heads / n_kv_heads) */
  int32_t head_dim;              /* 64 or 128 */
  int32_t page_size;             /* 16 */
  int64_t pool_pages;            /* pages in each pool */
  float scale;                   /* softmax scale; 0 means 1/sqrt(head_dim) */
} mx_attn_shape;

typedef struct {
  int32_t hidden; /* H, a multiple of 64 */
  int32_t ffn;    /* F, a multiple of 64 */
  mx_attn_shape attn;
  float rms_eps;    /* RMSNorm epsilon */
  float rope_theta; /* RoPE base (rotate-half pairing) */
} mx_layer_cfg;

/* Canonical weights, bf16, row-major [out][in] (the layout of a linear layer):
 *   ln1_g[H], w_qkv[(nq + 2 nkv) d][H] (rows: q heads, then k heads, then v heads),
 *   w_o[H][nq d], ln2_g[H], w_gate_up[2F][H] (rows: gate, then up), w_down[H][F]. */
typedef struct {
  const uint16_t *ln1_g, *w_qkv, *w_o, *ln2_g, *w_gate_up, *w_down;
} mx_layer_weights;

const char* mx_status_str(mx_status s);
/* Detail of the last error on the calling thread ("" if none). */
const char* mx_last_error(void);
/* ABI version: (major << 16) | minor. */
uint32_t mx_version(void);

/*
 * Host-only check of a batch against a shape (the rules every entry point
 * applies first): R >= 0; phase in {PREFILL, DECODE}; n_new >= 1; a decode has
 * n_new == 1 and ctx_len >= 1; ctx_len >= 0; n_pages >= ceil((ctx_len + n_new)/16)
 * (else MX_ERR_NO_SPACE); page ids in [0, pool_pages); the slots written by the
 * new tokens are distinct across the batch (cached prefix pages may be shared
 * read-only); n_q_heads % n_kv_heads == 0; head_dim in {64, 128} and
 * page_size == 16 (else MX_ERR_UNSUPPORTED).  Touches no device.
 */
mx_status mx_batch_validate(const mx_batch* batch, const mx_attn_shape* shape);

/*
 * Workspace bytes that a call needs for this batch (mx_layer_step when cfg is
 * given, mx_paged_attn / mx_kv_append when cfg is NULL and shape is given).
 * Returns 0 and sets mx_last_error on an invalid batch.
 */
size_t mx_workspace_bytes_for(const mx_batch* batch, const mx_attn_shape* shape,
                              const mx_layer_cfg* cfg);

/*
 * Upper bound of the workspace of mx_layer_step for any batch of at most
 * max_tokens new tokens, max_reqs requests and max_pages page-table entries in
 * total.  With cfg == NULL the bound for mx_paged_attn / mx_kv_append, using
 * shape.
 */
size_t mx_workspace_bytes(const mx_layer_cfg* cfg, const mx_attn_shape* shape,
                          int32_t max_tokens, int32_t max_reqs, int64_t max_pages);

/* Bytes of the packed weight blob of one layer. */
size_t mx_packed_weights_bytes(const mx_layer_cfg* cfg);

/*
 * Re-lays the canonical weights into the packed blob (device, packed_bytes
 * from mx_packed_weights_bytes) that mx_layer_step reads: the gate and up
 * rows of w_gate_up are interleaved in 32-row blocks so that one GEMM tile
 * holds both operands of the SwiGLU product, and within every q and k head of
 * w_qkv (head_dim 128) the rows of dims i and i + 64 are placed 32 rows apart
 * so that one lane holds both halves of each rotary pair.  Enqueued on the
 * stream.
 */
mx_status mx_pack_weights(const mx_layer_cfg* cfg, const mx_layer_weights* canonical,
                          void* packed, size_t packed_bytes, hipStream_t stream);

/*
 * KV append (the cache write of the new tokens).  The evaluation's serving
 * engine keeps keys and values in a paged cache (paper Section 5.1, the
 * vLLM-based engine and its baselines); the new tokens' keys and values enter
 * it before attention reads them.  k_new, v_new [T][n_kv_heads][head_dim] are
 * copied to the slots of the token map, k into k_pool's layout and v into
 * v_pool's transposed page layout.  A pure byte copy: the pools are bit-equal
 * to what a plain copy would leave.  Errors as every entry point: host checks
 * first (MX_ERR_NULL for a NULL tensor, MX_ERR_INVALID for a misaligned one,
 * MX_ERR_TOO_LARGE for a short workspace), nothing enqueued on error.
 */
mx_status mx_kv_append(const mx_batch* batch, const mx_attn_shape* shape,
                       const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                       uint16_t* v_pool, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Paged varlen attention over the mixed batch, one launch for prefill rows
 * and decode rows (paper Section 4.2 and Section 4.3: prefill chunks
 * piggybacked on decodes; Section 5.1: the paged cache of the vLLM-based engine):
 * q [T][n_q_heads][head_dim] -> out [T][n_q_heads][head_dim], bf16.  For token
 * t (request r, position p) and q head h, with g = h / (nq / nkv):
 *   out[t][h] = sum_{j <= p} softmax_j(scale * q[t][h] . K_r[j][g]) V_r[j][g],
 * K_r[j] and V_r[j] read from the pools through the request's page table.
 * Keys of positions 0 .. ctx_len + n_new - 1 must already be in the pools
 * (mx_kv_append puts the new ones there).  Slots at or beyond that length are
 * never read into a sum.  Long decode contexts are split across workgroups
 * and merged deterministically: results are bit-identical from run to run.
 */
mx_status mx_paged_attn(const mx_batch* batch, const mx_attn_shape* shape, const uint16_t* q,
                        const uint16_t* k_pool, const uint16_t* v_pool, uint16_t* out,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * mx_paged_attn without a workspace, for callers that cannot allocate device
 * memory (tight serving loops, harnesses that forbid hipMalloc): the same
 * kernels and the same results, bit for bit, with the call's metadata and
 * split partials in a static device array of mx_paged_attn_static_max_bytes()
 * bytes (32 MiB) that the library holds on every GPU it runs on until the
 * process ends.  Allocates no device or pinned memory (the host-side plan
 * uses ordinary heap memory): the metadata is packed into a static host buffer
 * of the library and copied into the array with hipMemcpyAsync on the stream,
 * which HIP performs synchronously from pageable memory (the call returns once
 * the copy has run).  The copy reads that host buffer when it runs, so the
 * call is not meant for HIP graph capture (a captured copy would read
 * whatever a later call packed there).  A batch whose metadata and partials
 * need more than the array holds returns MX_ERR_TOO_LARGE before any device
 * work.  All calls on one GPU share that GPU's array: calls that overlap on one
 * GPU (different streams, or threads without ordering) race; calls ordered on
 * one stream do not.  Other errors as mx_paged_attn.
 */
size_t mx_paged_attn_static_max_bytes(void);
mx_status mx_paged_attn_static(const mx_batch* batch, const mx_attn_shape* shape, const uint16_t* q,
                               const uint16_t* k_pool, const uint16_t* v_pool, uint16_t* out,
                               hipStream_t stream);

/*
 * One multiplexed decoder-layer iteration: a multiplexing worker's iteration
 * in which the prefill chunks the toggle piggybacks onto the running decode
 * batch (paper Section 4.2, "SLO-Aware Multiplexing", and Section 4.3,
 * "Multiplexing Toggle"; one chunk per iteration, Section 5.1) pass through
 * the layer together with the decodes.  Its latency as a function of the
 * prefill tokens mixed in is the interference the toggle prices against the
 * decodes' TPOT slack (Section 4.2).  The paper states no layer arithmetic; the
 * layer is the pre-norm Llama-style layer of the benchmark shapes:
 *   h  = RMSNorm(x) * ln1_g
 *   q, k, v = h W_qkv^T;  RoPE (rotate-half, base rope_theta) on q and k at
 *             each token's position
 *   k, v -> pools (append), then attention as mx_paged_attn -> o
 *   x1 = x + o W_o^T
 *   h2 = RMSNorm(x1) * ln2_g
 *   a  = silu(h2 W_gate^T) * (h2 W_up^T)
 *   y  = x1 + a W_down^T
 * x, y [T][H] bf16 (y must not alias x); packed_weights from mx_pack_weights.
 * Repeating a call with the same inputs rewrites the same slots with the same
 * values.
 */
mx_status mx_layer_step(const mx_batch* batch, const mx_layer_cfg* cfg, const void* packed_weights,
                        const uint16_t* x, uint16_t* y, uint16_t* k_pool, uint16_t* v_pool,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- inspection */

/* Byte offsets, inside the workspace of mx_layer_step for this batch, of the
 * intermediate tensors the call leaves behind (bf16):
 *   off[0] h / h2 [T][H] (h2 overwrites h), off[1] q [T][nq][d] (post-RoPE),
 *   off[2] o [T][nq * d], off[3] x1 [T][H], off[4] a [T][F].
 * q and x1 are row-major.  h, o and a, the inputs of the projections, are in
 * the projection-input tile layout: a T x K matrix stored as ceil(T / 16) tile
 * rows, each K / 32 tiles of 16 rows x 32 columns (one contiguous kilobyte)
 * followed by one unused tile, element (t, c) at
 *   (t / 16) * (16 * K + 512) + (c / 32) * 512 + (t % 16) * 32 + c % 32,
 * ceil(T / 16) * (16 * K + 512) elements in all (the GEMMs copy whole
 * kilobytes, as they do from the packed weights; the unused tile keeps tile
 * rows off power-of-two distances).
 * (The new keys and values of the iteration are in the pools.) */
mx_status mx_layer_workspace_offsets(const mx_batch* batch, const mx_layer_cfg* cfg,
                                     size_t off[5]);

/* Device token map of the batch as the iteration computes it (the kernel that
 * every entry point runs first): tok_req[T], tok_pos[T] (int32) and
 * tok_slot[T] (int64), device outputs. */
mx_status mx_debug_token_map(const mx_batch* batch, const mx_attn_shape* shape, int32_t* tok_req,
                             int32_t* tok_pos, int64_t* tok_slot, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/* Gathers request req's keys and values, positions 0 .. ctx_len + n_new - 1, from
 * the pools through its page table into k_out, v_out [len][n_kv_heads][head_dim]
 * (device).  A byte copy through the same addressing the attention uses. */
mx_status mx_debug_gather(const mx_batch* batch, const mx_attn_shape* shape, int32_t req,
                          const uint16_t* k_pool, const uint16_t* v_pool, uint16_t* k_out,
                          uint16_t* v_out, void* ws, size_t ws_bytes, hipStream_t stream);

/* Launch timing, for profiling.  When enabled, every kernel launch of
 * mx_layer_step and mx_paged_attn is bracketed by two hipEvents recorded on the
 * caller's stream (the launch's own stream), tagged with the step it performs
 * ("token_map+rmsnorm_1", "gemm_qkv", "paged_attn", "gemm_o", "rmsnorm_2",
 * "gemm_gate_up", "gemm_down"; a tag covers a split-K GEMM's reduce, the
 * launches of a GEMM whose rows run as two parts, and the attention's split
 * merge, except that when rows of the output projection are split over K their
 * reduce runs fused with the second RMSNorm, timed as "o_reduce+rmsnorm_2"
 * instead of "rmsnorm_2").  Off by default. */
mx_status mx_profile_enable(int32_t on);
/* Waits for the recorded events, accumulates their durations per tag and
 * returns the number of tags written (at most max_entries): names[i] is a
 * static string, total_ms[i] the summed duration and counts[i] the number of
 * launches.  Clears what it reports.  Any output array may be NULL. */
int32_t mx_profile_read(const char** names, float* total_ms, int32_t* counts, int32_t max_entries);

/* The projection GEMM of the layer on its own: C[M][N] = epi(A[M][K] B[N][K]^T),
 * bf16 in, fp32 accumulate; epilogue 0 = store, 1 = + R[M][N] (residual),
 * 2 = SwiGLU over B rows interleaved gate/up in 32-row blocks (C is [M][N/2]).
 * R must not overlap C.  K must be a multiple of 64.  ws holds the K-split scratch
 * (mx_debug_gemm_ws_bytes).  For tests and microbenchmarks. */
size_t mx_debug_gemm_ws_bytes(int32_t M, int32_t N, int32_t K);
mx_status mx_debug_gemm(int32_t M, int32_t N, int32_t K, const uint16_t* A, const uint16_t* B,
                        uint16_t* C, const uint16_t* R, int32_t epilogue, void* ws, size_t ws_bytes,
                        hipStream_t stream);
/* The same with a forced tile shape (0: 256x256, 1: 128x256, 2: 128x128, 3: 64x128,
 * 4: 128x256 with a shallower LDS ring, two workgroups per CU;
 * -1: the library's own choice) and K split: 1 <= ksplit <= min(64, K / 64), else
 * MX_ERR_INVALID; split z takes the 64-wide K chunks [z C / ksplit, (z + 1) C / ksplit)
 * of the C = K / 64, so ksplit need not divide C.  ws must hold ksplit * M * N floats
 * when ksplit > 1.  For tuning sweeps. */
mx_status mx_debug_gemm_config(int32_t M, int32_t N, int32_t K, const uint16_t* A, const uint16_t* B,
                               uint16_t* C, const uint16_t* R, int32_t epilogue, int32_t tile_cfg,
                               int32_t ksplit, void* ws, size_t ws_bytes, hipStream_t stream);
/* The same with every operand in the layer step's own layout: B in the packed-weight
 * tile layout, element (n, k) at ((n / 16) * (K / 32) + k / 32) * 512 + (n % 16) * 32
 * + k % 32, i.e. 16 x 32 tiles of 1 KB ordered [N / 16][K / 32]; A in the projection-input
 * tile layout of mx_layer_workspace_offsets over its M rows (ceil(M / 16) * (16 * K + 512)
 * elements; the padding rows of the last tile row and the unused tiles are never read);
 * C row-major [M][N], except the SwiGLU output, which is in that tile layout too (with
 * N / 2 columns; the padding rows and unused tiles are never written), as the layer's
 * down projection reads it.  R row-major.  N % 16 == 0 and
 * K % 32 == 0 (else MX_ERR_UNSUPPORTED).  For tests and tuning sweeps of the layer's
 * own operand layout. */
mx_status mx_debug_gemm_tiled(int32_t M, int32_t N, int32_t K, const uint16_t* A,
                              const uint16_t* B_tiled, uint16_t* C, const uint16_t* R,
                              int32_t epilogue, int32_t tile_cfg, int32_t ksplit, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/* The tile plan the library's cost model picks for an M x N x K projection
 * (host only, touches no device): plan[0] tile shape (numbered as for
 * mx_debug_gemm_config) and plan[1] K split of rows [0, plan[2]); when
 * plan[2] < M the remaining rows run as a second GEMM after the first, with
 * tile shape plan[3] and K split plan[4] (plan[2] == M: one launch, plan[3] = -1).
 * K must be a multiple of 64.  For tests that must know which path a shape takes. */
mx_status mx_debug_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t plan[5]);
/* A forced row split with the operands in the layer's layouts (as
 * mx_debug_gemm_tiled): rows [0, m_main) with tile shape main_cfg and no K split,
 * then rows [m_main, M) as a GEMM of their own with tile shape tail_cfg and K split
 * tail_ksplit (ws holds tail_ksplit * (M - m_main) * N floats when it is > 1).
 * 1 <= m_main < M with m_main % 16 == 0 (the second GEMM starts a tile row),
 * N % 16 == 0, K % 64 == 0.  For tests of the row split. */
mx_status mx_debug_gemm_rows(int32_t M, int32_t N, int32_t K, const uint16_t* A,
                             const uint16_t* B_tiled, uint16_t* C, const uint16_t* R,
                             int32_t epilogue, int32_t m_main, int32_t main_cfg, int32_t tail_cfg,
                             int32_t tail_ksplit, void* ws, size_t ws_bytes, hipStream_t stream);
/* The output projection's split-K reduce fused with the second RMSNorm, on its
 * own: for rows r >= split_row, x1[r] = bf16(sum_z partial[z][r - split_row] + R[r])
 * (partial: ksplit fp32 planes [M - split_row][H], summed in plane order, then
 * the residual); rows r < split_row hold x1 already.  Then h[r] = RMSNorm(x1[r]) * g
 * for every row, from the rounded x1.  R, x1 [M][H] bf16 row-major, g [H] bf16, h
 * in the projection-input tile layout (mx_layer_workspace_offsets; ceil(M / 16) *
 * (16 * H + 512) elements); H % 32 == 0 and H <= 8192.  For tests of the kernel the layer step
 * runs. */
mx_status mx_debug_reduce_residual_rmsnorm(const float* partial, int32_t ksplit, const uint16_t* R,
                                           uint16_t* x1, const uint16_t* g, uint16_t* h, int32_t M,
                                           int32_t H, float eps, int32_t split_row,
                                           hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif
