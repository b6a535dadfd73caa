/*
 * oracle.h -- plain, slow, fp64 CPU reference of one multiplexed decoder-layer
 * iteration (prefill chunks co-batched with single-token decodes over a paged
 * KV cache).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this code; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or helper with the
 * HIP path.
 *
 * What the paper fixes and what it does not.  The paper (Section 4.3, "Multiplexing
 * Toggle", and Section 5.1, "Experimental Setup") describes a worker iteration in
 * which chunked prefill requests are piggybacked onto the running decode batch,
 * served by a vLLM-style engine with a paged KV cache.  It states no layer
 * arithmetic.  The layer computed here is the textbook pre-norm decoder layer
 * (RMSNorm -> QKV projection -> RoPE -> causal softmax attention -> output
 * projection + residual -> RMSNorm -> SwiGLU MLP + residual); every choice the
 * paper leaves open is listed in the repository's design notes.
 *
 * Precision: every floating-point value is held and computed in IEEE double.
 * Inputs that the workload defines in bfloat16 (activations, weights, cached
 * keys/values) are passed as raw bf16 bit patterns and widened exactly.
 *
 * Threading: loops over independent rows use OpenMP when compiled with it;
 * each output element is computed by one thread in a fixed order, so results
 * do not depend on the thread count.
 *
 * Parity pins: every function below is checked by the CPU test suite against
 * closed forms, invariants, brute force or an independent library routine
 * (numpy / torch CPU in float64).
 */
#ifndef MX_ORACLE_H
#define MX_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Exact widening of a bfloat16 bit pattern. */
double orc_bf16_to_double(uint16_t bits);

/* Number of OpenMP threads the oracle's parallel loops use (1 without OpenMP). */
int orc_num_threads(void);

/*
 * Token map of a mixed batch (the per-request fields a scheduler hands to a
 * worker: new-token count, cached context length, page table).
 * Request r owns tokens [cu_q[r], cu_q[r+1]) of the concatenated batch; its
 * i-th new token sits at position ctx_len[r] + i and is written to KV slot
 *   pages[page_off[r] + pos / page_size] * page_size + pos % page_size.
 * pages is the concatenation of the per-request page tables, request r's
 * table being pages[page_off[r] .. page_off[r+1]).
 * Returns 0, or -1 if a request's page table is too short for its positions.
 */
int orc_token_map(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                  const int64_t* page_off, const int32_t* pages, int32_t page_size,
                  int32_t* cu_q, int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot);

/* out[t][i] = x[t][i] / sqrt(mean_i x[t][i]^2 + eps) * g[i] */
void orc_rmsnorm(int64_t T, int64_t H, const double* x, const double* g, double eps,
                 double* out);

/* out[t][n] = sum_k a[t][k] * W[n][k]; W is row-major [N][K] (bf16 bits). */
void orc_linear(int64_t T, int64_t K, int64_t N, const double* a, const uint16_t* W,
                double* out);

/*
 * Rotary position embedding, rotate-half pairing, in place on u[T][nheads][d]:
 * for i < d/2, angle = pos[t] * theta^(-2i/d),
 *   (u_i, u_{i+d/2}) <- (u_i cos - u_{i+d/2} sin, u_{i+d/2} cos + u_i sin).
 */
void orc_rope(int64_t T, int32_t nheads, int32_t d, const int32_t* pos, double theta,
              double* u);

/* a[t][f] = silu(gu[t][f]) * gu[t][F + f], silu(z) = z / (1 + exp(-z)). */
void orc_silu_mul(int64_t T, int64_t F, const double* gu, double* a);

/*
 * Causal softmax attention for a mixed batch, keys/values held per request in
 * contiguous arrays.  Request r's keys for positions 0..kv_len-1 are
 *   kc[(kv_off[r] + j) * nkv * d + g * d + i]  (same for vc),
 * kv_len = ctx_len[r] + n_new[r].  Token t = cu_q[r] + i (position p =
 * ctx_len[r] + i) and query head h (kv head g = h / (nq / nkv)) produce
 *   o[t][h] = sum_{j<=p} softmax_j(scale * q[t][h] . k_j) v_j.
 * q and o are [T][nq][d].
 */
void orc_attention_contig(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                          int32_t nq, int32_t nkv, int32_t d, double scale,
                          const double* q, const double* kc, const double* vc,
                          const int64_t* kv_off, double* o);

/*
 * The same attention, with keys/values gathered from a paged pool laid out
 * [pool_pages][nkv][page_size][d] through per-request page tables (same
 * convention as orc_token_map).  Arithmetic and loop order are those of
 * orc_attention_contig, so the two agree bit for bit when the pool holds the
 * same values.  Returns 0, or -1 on a page id outside [0, pool_pages).
 */
int orc_attention_paged(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                        int32_t nq, int32_t nkv, int32_t d, double scale,
                        const double* q, const double* k_pool, const double* v_pool,
                        int64_t pool_pages, int32_t page_size,
                        const int64_t* page_off, const int32_t* pages, double* o);

/*
 * Normalised attention weights of one (token, query head) of the contiguous
 * variant: w[j] for j = 0..p.  Used by tests to check that each softmax row
 * sums to one.  Returns the number of weights written (p + 1).
 */
int64_t orc_attention_weights(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                              int32_t nq, int32_t nkv, int32_t d, double scale,
                              const double* q, const double* kc, const int64_t* kv_off,
                              int64_t t, int32_t h, double* w);

typedef struct {
  int32_t hidden, ffn, n_q_heads, n_kv_heads, head_dim;
  double rms_eps, rope_theta, scale;
} orc_layer_cfg;

/*
 * One multiplexed decoder-layer iteration over a mixed batch.
 *
 * Inputs (bf16 bit patterns):
 *   x[T][H]                     token activations, request-major;
 *   g1[H], w_qkv[(nq+2nkv)d][H], w_o[H][nq d], g2[H], w_gu[2F][H], w_down[H][F]
 *                               weights, rows of w_qkv ordered q heads, k heads,
 *                               v heads; rows of w_gu ordered gate, then up;
 *   k_prior, v_prior            cached keys/values of positions < ctx_len[r],
 *                               [sum_r ctx_len[r]][nkv][d], request-major
 *                               (these are post-RoPE values and are not rotated
 *                               again).
 * rows: ascending token indices at which the attention and everything after it
 *   is evaluated (n_rows of them), or NULL to evaluate all T rows.  Keys and
 *   values of every token are always computed, since later rows need them.
 * Outputs (double):
 *   h[T][H]          RMSNorm-1 output, all tokens;
 *   k_new, v_new     [T][nkv][d], post-RoPE keys and values of all new tokens;
 *   q[n_rows][nq][d] post-RoPE queries; o[n_rows][nq d] attention output;
 *   x1[n_rows][H], h2[n_rows][H], a[n_rows][F], y[n_rows][H].
 * Any output pointer may be NULL except k_new and v_new.
 * Returns 0 on success, -1 on an invalid argument.
 */
int orc_layer_step(const orc_layer_cfg* cfg, int32_t R, const int32_t* n_new,
                   const int32_t* ctx_len, const uint16_t* x, const uint16_t* g1,
                   const uint16_t* w_qkv, const uint16_t* w_o, const uint16_t* g2,
                   const uint16_t* w_gu, const uint16_t* w_down, const uint16_t* k_prior,
                   const uint16_t* v_prior, int64_t n_rows, const int64_t* rows,
                   double* h, double* k_new, double* v_new, double* q, double* o,
                   double* x1, double* h2, double* a, double* y);

/*
 * Append new keys/values (bf16 bits, [T][nkv][d]) into paged pools
 * ([pool_pages][nkv][page_size][d], bf16 bits) at the slots of orc_token_map.
 * A pure byte copy.  Returns 0, or -1 on a page table that is too short or a
 * page id outside the pool.
 */
int orc_kv_append(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                  const int64_t* page_off, const int32_t* pages, int32_t page_size,
                  int32_t nkv, int32_t d, const uint16_t* k_new, const uint16_t* v_new,
                  uint16_t* k_pool, uint16_t* v_pool, int64_t pool_pages);

#ifdef __cplusplus
}
#endif
#endif
