/*
 * oracle.c -- plain fp64 CPU reference of one multiplexed decoder-layer
 * iteration.  TEST INFRASTRUCTURE ONLY: only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark use it; the product library never does.
 *
 * Each function follows the plain mathematical definition of its step, written
 * out without blocking, fusion or reordering.  The per-function comments name
 * the passage of the paper that puts the step on the path; the arithmetic of
 * each step is the textbook definition because the paper states none.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

double orc_bf16_to_double(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/*
 * Mixed batch bookkeeping (Section 4.3: prefill chunks are piggybacked onto the
 * decode requests of a multiplexing worker; Section 5.1: the engine keeps a paged
 * KV cache).  Tokens are concatenated in request order.
 */
int orc_token_map(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                  const int64_t* page_off, const int32_t* pages, int32_t page_size,
                  int32_t* cu_q, int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot) {
  cu_q[0] = 0;
  for (int32_t r = 0; r < R; r++) cu_q[r + 1] = cu_q[r] + n_new[r];
  for (int32_t r = 0; r < R; r++) {
    int64_t table_len = page_off[r + 1] - page_off[r];
    for (int32_t i = 0; i < n_new[r]; i++) {
      int32_t t = cu_q[r] + i;
      int32_t p = ctx_len[r] + i;
      int64_t page_index = p / page_size;
      if (page_index >= table_len) return -1;
      tok_req[t] = r;
      tok_pos[t] = p;
      tok_slot[t] = (int64_t)pages[page_off[r] + page_index] * page_size + p % page_size;
    }
  }
  return 0;
}

/* Root-mean-square normalisation with a learned gain. */
void orc_rmsnorm(int64_t T, int64_t H, const double* x, const double* g, double eps,
                 double* out) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; t++) {
    const double* xr = x + t * H;
    double ss = 0.0;
    for (int64_t i = 0; i < H; i++) ss += xr[i] * xr[i];
    double inv = 1.0 / sqrt(ss / (double)H + eps);
    for (int64_t i = 0; i < H; i++) out[t * H + i] = xr[i] * inv * g[i];
  }
}

/* Dense projection out = a W^T with W stored [N][K]. */
void orc_linear(int64_t T, int64_t K, int64_t N, const double* a, const uint16_t* W,
                double* out) {
#pragma omp parallel
  {
    double* wrow = (double*)malloc((size_t)K * sizeof(double));
#pragma omp for schedule(static)
    for (int64_t n = 0; n < N; n++) {
      for (int64_t k = 0; k < K; k++) wrow[k] = orc_bf16_to_double(W[n * K + k]);
      for (int64_t t = 0; t < T; t++) {
        const double* ar = a + t * K;
        double s = 0.0;
        for (int64_t k = 0; k < K; k++) s += ar[k] * wrow[k];
        out[t * N + n] = s;
      }
    }
    free(wrow);
  }
}

/* Rotary position embedding with the rotate-half pairing. */
void orc_rope(int64_t T, int32_t nheads, int32_t d, const int32_t* pos, double theta,
              double* u) {
  int32_t half = d / 2;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; t++) {
    for (int32_t hd = 0; hd < nheads; hd++) {
      double* v = u + (t * nheads + hd) * d;
      for (int32_t i = 0; i < half; i++) {
        double angle = (double)pos[t] * pow(theta, -2.0 * (double)i / (double)d);
        double c = cos(angle), s = sin(angle);
        double a0 = v[i], a1 = v[i + half];
        v[i] = a0 * c - a1 * s;
        v[i + half] = a1 * c + a0 * s;
      }
    }
  }
}

/* SwiGLU gating: silu(gate) * up. */
void orc_silu_mul(int64_t T, int64_t F, const double* gu, double* a) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; t++) {
    for (int64_t f = 0; f < F; f++) {
      double g = gu[t * 2 * F + f];
      double up = gu[t * 2 * F + F + f];
      a[t * F + f] = g / (1.0 + exp(-g)) * up;
    }
  }
}

/*
 * Softmax attention of one query row over n keys given by row pointers:
 * s_j = scale * q.k_j, w_j = exp(s_j - max s), o = sum_j w_j v_j / sum_j w_j.
 * Both the contiguous and the paged variant call this, so they differ only in
 * how the key/value rows are located.
 */
static void attend_row(int32_t d, double scale, const double* qv, int64_t n,
                       const double* const* krow, const double* const* vrow, double* w,
                       double* out, int normalise_weights) {
  double m = -INFINITY;
  for (int64_t j = 0; j < n; j++) {
    double s = 0.0;
    for (int32_t i = 0; i < d; i++) s += qv[i] * krow[j][i];
    s *= scale;
    w[j] = s;
    if (s > m) m = s;
  }
  double l = 0.0;
  for (int64_t j = 0; j < n; j++) {
    w[j] = exp(w[j] - m);
    l += w[j];
  }
  if (out) {
    for (int32_t i = 0; i < d; i++) out[i] = 0.0;
    for (int64_t j = 0; j < n; j++)
      for (int32_t i = 0; i < d; i++) out[i] += w[j] * vrow[j][i];
    for (int32_t i = 0; i < d; i++) out[i] /= l;
  }
  if (normalise_weights)
    for (int64_t j = 0; j < n; j++) w[j] /= l;
}

/* Row pointers of request r's keys (and values) for positions 0..n-1. */
typedef struct {
  int paged;
  int32_t nkv, d, page_size;
  const double *k, *v;         /* contiguous arrays or pools */
  int64_t kv_off;              /* contiguous: token offset of the request */
  const int32_t* table;        /* paged: the request's page table */
  int64_t pool_pages;
} kv_source;

static int kv_rows(const kv_source* src, int32_t g, int64_t n, const double** krow,
                   const double** vrow) {
  for (int64_t j = 0; j < n; j++) {
    int64_t base;
    if (src->paged) {
      int64_t page = src->table[j / src->page_size];
      if (page < 0 || page >= src->pool_pages) return -1;
      base = ((page * src->nkv + g) * src->page_size + j % src->page_size) * src->d;
    } else {
      base = ((src->kv_off + j) * src->nkv + g) * src->d;
    }
    krow[j] = src->k + base;
    vrow[j] = src->v ? src->v + base : NULL;
  }
  return 0;
}

/* Longest key sequence of the batch, for scratch sizing. */
static int64_t max_kv_len(int32_t R, const int32_t* n_new, const int32_t* ctx_len) {
  int64_t m = 1;
  for (int32_t r = 0; r < R; r++)
    if ((int64_t)ctx_len[r] + n_new[r] > m) m = (int64_t)ctx_len[r] + n_new[r];
  return m;
}

/* Causal attention of every (token, query head) of the batch; see the header. */
static int attention_batch(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                           int32_t nq, int32_t nkv, int32_t d, double scale,
                           const double* q, kv_source base, const int64_t* kv_off,
                           const int64_t* page_off, const int32_t* pages, double* o) {
  int32_t group = nq / nkv;
  int64_t nmax = max_kv_len(R, n_new, ctx_len);
  int64_t* first = (int64_t*)malloc((size_t)(R + 1) * sizeof(int64_t));
  first[0] = 0;
  for (int32_t r = 0; r < R; r++) first[r + 1] = first[r] + n_new[r];
  int64_t T = first[R];
  int failed = 0;
#pragma omp parallel
  {
    const double** krow = (const double**)malloc((size_t)nmax * sizeof(double*));
    const double** vrow = (const double**)malloc((size_t)nmax * sizeof(double*));
    double* w = (double*)malloc((size_t)nmax * sizeof(double));
#pragma omp for schedule(dynamic, 1)
    for (int64_t t = 0; t < T; t++) {
      int32_t r = 0;
      while (first[r + 1] <= t) r++;
      int64_t p = ctx_len[r] + (t - first[r]);
      kv_source src = base;
      if (src.paged)
        src.table = pages + page_off[r];
      else
        src.kv_off = kv_off[r];
      for (int32_t h = 0; h < nq; h++) {
        if (kv_rows(&src, h / group, p + 1, krow, vrow) != 0) {
#pragma omp atomic write
          failed = 1;
          break;
        }
        attend_row(d, scale, q + (t * nq + h) * d, p + 1, krow, vrow, w,
                   o + (t * nq + h) * d, 0);
      }
    }
    free(krow);
    free(vrow);
    free(w);
  }
  free(first);
  return failed ? -1 : 0;
}

/* Section 4.3 / Section 5.1: one attention launch serves the prefill rows and the
 * decode rows of the multiplexed batch. */
void orc_attention_contig(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                          int32_t nq, int32_t nkv, int32_t d, double scale,
                          const double* q, const double* kc, const double* vc,
                          const int64_t* kv_off, double* o) {
  kv_source src = {0, nkv, d, 0, kc, vc, 0, NULL, 0};
  attention_batch(R, n_new, ctx_len, nq, nkv, d, scale, q, src, kv_off, NULL, NULL, o);
}

int orc_attention_paged(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                        int32_t nq, int32_t nkv, int32_t d, double scale,
                        const double* q, const double* k_pool, const double* v_pool,
                        int64_t pool_pages, int32_t page_size,
                        const int64_t* page_off, const int32_t* pages, double* o) {
  for (int32_t r = 0; r < R; r++) {
    int64_t need = ((int64_t)ctx_len[r] + n_new[r] + page_size - 1) / page_size;
    if (page_off[r + 1] - page_off[r] < need) return -1;
  }
  kv_source src = {1, nkv, d, page_size, k_pool, v_pool, 0, NULL, pool_pages};
  return attention_batch(R, n_new, ctx_len, nq, nkv, d, scale, q, src, NULL, page_off,
                         pages, o);
}

int64_t orc_attention_weights(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                              int32_t nq, int32_t nkv, int32_t d, double scale,
                              const double* q, const double* kc, const int64_t* kv_off,
                              int64_t t, int32_t h, double* w) {
  int32_t r = 0;
  int64_t first = 0;
  while (r < R && first + n_new[r] <= t) first += n_new[r++];
  if (r >= R) return -1;
  int64_t p = ctx_len[r] + (t - first);
  kv_source src = {0, nkv, d, 0, kc, NULL, kv_off[r], NULL, 0};
  const double** krow = (const double**)malloc((size_t)(p + 1) * sizeof(double*));
  const double** vrow = (const double**)malloc((size_t)(p + 1) * sizeof(double*));
  kv_rows(&src, h / (nq / nkv), p + 1, krow, vrow);
  attend_row(d, scale, q + (t * nq + h) * d, p + 1, krow, vrow, w, NULL, 1);
  free(krow);
  free(vrow);
  return p + 1;
}

/* Widen a bf16 array. */
static double* widen(const uint16_t* src, int64_t n) {
  double* dst = (double*)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) dst[i] = orc_bf16_to_double(src[i]);
  return dst;
}

/*
 * The whole layer (see the header for the argument contract).  The steps are,
 * in order: token map; RMSNorm 1; K and V projections of every new token and
 * RoPE on K; Q projection and RoPE of the evaluated rows; causal attention of
 * the evaluated rows over cached plus new keys; output projection + residual;
 * RMSNorm 2; gate/up projection and SwiGLU; down projection + residual.
 */
int orc_layer_step(const orc_layer_cfg* c, int32_t R, const int32_t* n_new,
                   const int32_t* ctx_len, const uint16_t* x, const uint16_t* g1,
                   const uint16_t* w_qkv, const uint16_t* w_o, const uint16_t* g2,
                   const uint16_t* w_gu, const uint16_t* w_down, const uint16_t* k_prior,
                   const uint16_t* v_prior, int64_t n_rows, const int64_t* rows,
                   double* h_out, double* k_new, double* v_new, double* q_out, double* o_out,
                   double* x1_out, double* h2_out, double* a_out, double* y_out) {
  const int64_t H = c->hidden, F = c->ffn, nq = c->n_q_heads, nkv = c->n_kv_heads,
                d = c->head_dim;
  if (R < 0 || H <= 0 || F <= 0 || nq <= 0 || nkv <= 0 || d <= 0 || d % 2 || nq % nkv)
    return -1;
  if (!k_new || !v_new) return -1;

  /* token map (positions only; the layer needs no slots) */
  int32_t* cu_q = (int32_t*)malloc((size_t)(R + 1) * sizeof(int32_t));
  cu_q[0] = 0;
  for (int32_t r = 0; r < R; r++) {
    if (n_new[r] < 1 || ctx_len[r] < 0) { free(cu_q); return -1; }
    cu_q[r + 1] = cu_q[r] + n_new[r];
  }
  const int64_t T = cu_q[R];
  int32_t* pos = (int32_t*)malloc((size_t)(T > 0 ? T : 1) * sizeof(int32_t));
  int32_t* req = (int32_t*)malloc((size_t)(T > 0 ? T : 1) * sizeof(int32_t));
  for (int32_t r = 0; r < R; r++)
    for (int32_t i = 0; i < n_new[r]; i++) {
      pos[cu_q[r] + i] = ctx_len[r] + i;
      req[cu_q[r] + i] = r;
    }
  int64_t nr = rows ? n_rows : T;
  int64_t* row_idx = (int64_t*)malloc((size_t)(nr > 0 ? nr : 1) * sizeof(int64_t));
  for (int64_t i = 0; i < nr; i++) {
    row_idx[i] = rows ? rows[i] : i;
    if (row_idx[i] < 0 || row_idx[i] >= T) {
      free(cu_q); free(pos); free(req); free(row_idx);
      return -1;
    }
  }

  /* RMSNorm 1 over every token */
  double* xd = widen(x, T * H);
  double* g1d = widen(g1, H);
  double* h = (double*)malloc((size_t)(T * H > 0 ? T * H : 1) * sizeof(double));
  orc_rmsnorm(T, H, xd, g1d, c->rms_eps, h);

  /* K, V projections of every new token (w_qkv rows: q heads, k heads, v heads) */
  orc_linear(T, H, nkv * d, h, w_qkv + nq * d * H, k_new);
  orc_linear(T, H, nkv * d, h, w_qkv + (nq + nkv) * d * H, v_new);
  orc_rope(T, (int32_t)nkv, (int32_t)d, pos, c->rope_theta, k_new);

  /* Q projection of the evaluated rows */
  double* hr = (double*)malloc((size_t)(nr * H > 0 ? nr * H : 1) * sizeof(double));
  int32_t* pos_r = (int32_t*)malloc((size_t)(nr > 0 ? nr : 1) * sizeof(int32_t));
  for (int64_t i = 0; i < nr; i++) {
    memcpy(hr + i * H, h + row_idx[i] * H, (size_t)H * sizeof(double));
    pos_r[i] = pos[row_idx[i]];
  }
  double* q = (double*)malloc((size_t)(nr * nq * d > 0 ? nr * nq * d : 1) * sizeof(double));
  orc_linear(nr, H, nq * d, hr, w_qkv, q);
  orc_rope(nr, (int32_t)nq, (int32_t)d, pos_r, c->rope_theta, q);

  /* Per-request contiguous K/V: cached prefix followed by the new tokens. */
  int64_t* kv_off = (int64_t*)malloc((size_t)(R + 1) * sizeof(int64_t));
  int64_t* prior_off = (int64_t*)malloc((size_t)(R + 1) * sizeof(int64_t));
  kv_off[0] = 0;
  prior_off[0] = 0;
  for (int32_t r = 0; r < R; r++) {
    kv_off[r + 1] = kv_off[r] + ctx_len[r] + n_new[r];
    prior_off[r + 1] = prior_off[r] + ctx_len[r];
  }
  int64_t row_elems = nkv * d;
  double* kc = (double*)malloc((size_t)(kv_off[R] * row_elems > 0 ? kv_off[R] * row_elems : 1) * sizeof(double));
  double* vc = (double*)malloc((size_t)(kv_off[R] * row_elems > 0 ? kv_off[R] * row_elems : 1) * sizeof(double));
  for (int32_t r = 0; r < R; r++) {
    for (int64_t j = 0; j < ctx_len[r]; j++)
      for (int64_t e = 0; e < row_elems; e++) {
        kc[(kv_off[r] + j) * row_elems + e] = orc_bf16_to_double(k_prior[(prior_off[r] + j) * row_elems + e]);
        vc[(kv_off[r] + j) * row_elems + e] = orc_bf16_to_double(v_prior[(prior_off[r] + j) * row_elems + e]);
      }
    for (int64_t i = 0; i < n_new[r]; i++)
      for (int64_t e = 0; e < row_elems; e++) {
        kc[(kv_off[r] + ctx_len[r] + i) * row_elems + e] = k_new[(cu_q[r] + i) * row_elems + e];
        vc[(kv_off[r] + ctx_len[r] + i) * row_elems + e] = v_new[(cu_q[r] + i) * row_elems + e];
      }
  }

  /* Attention of the evaluated rows: each row is its own single-token
   * "request" whose cached context is everything at or before its position. */
  int32_t* row_n = (int32_t*)malloc((size_t)(nr > 0 ? nr : 1) * sizeof(int32_t));
  int32_t* row_ctx = (int32_t*)malloc((size_t)(nr > 0 ? nr : 1) * sizeof(int32_t));
  int64_t* row_off = (int64_t*)malloc((size_t)(nr > 0 ? nr : 1) * sizeof(int64_t));
  for (int64_t i = 0; i < nr; i++) {
    row_n[i] = 1;
    row_ctx[i] = pos_r[i];
    row_off[i] = kv_off[req[row_idx[i]]];
  }
  double* o = (double*)malloc((size_t)(nr * nq * d > 0 ? nr * nq * d : 1) * sizeof(double));
  orc_attention_contig((int32_t)nr, row_n, row_ctx, (int32_t)nq, (int32_t)nkv, (int32_t)d,
                       c->scale, q, kc, vc, row_off, o);

  /* output projection + residual */
  double* x1 = (double*)malloc((size_t)(nr * H > 0 ? nr * H : 1) * sizeof(double));
  orc_linear(nr, nq * d, H, o, w_o, x1);
  for (int64_t i = 0; i < nr; i++)
    for (int64_t e = 0; e < H; e++) x1[i * H + e] += xd[row_idx[i] * H + e];

  /* RMSNorm 2, gate/up, SwiGLU, down + residual */
  double* g2d = widen(g2, H);
  double* h2 = (double*)malloc((size_t)(nr * H > 0 ? nr * H : 1) * sizeof(double));
  orc_rmsnorm(nr, H, x1, g2d, c->rms_eps, h2);
  double* gu = (double*)malloc((size_t)(nr * 2 * F > 0 ? nr * 2 * F : 1) * sizeof(double));
  orc_linear(nr, H, 2 * F, h2, w_gu, gu);
  double* a = (double*)malloc((size_t)(nr * F > 0 ? nr * F : 1) * sizeof(double));
  orc_silu_mul(nr, F, gu, a);
  double* y = (double*)malloc((size_t)(nr * H > 0 ? nr * H : 1) * sizeof(double));
  orc_linear(nr, F, H, a, w_down, y);
  for (int64_t i = 0; i < nr * H; i++) y[i] += x1[i];

  if (h_out) memcpy(h_out, h, (size_t)(T * H) * sizeof(double));
  if (q_out) memcpy(q_out, q, (size_t)(nr * nq * d) * sizeof(double));
  if (o_out) memcpy(o_out, o, (size_t)(nr * nq * d) * sizeof(double));
  if (x1_out) memcpy(x1_out, x1, (size_t)(nr * H) * sizeof(double));
  if (h2_out) memcpy(h2_out, h2, (size_t)(nr * H) * sizeof(double));
  if (a_out) memcpy(a_out, a, (size_t)(nr * F) * sizeof(double));
  if (y_out) memcpy(y_out, y, (size_t)(nr * H) * sizeof(double));

  free(cu_q); free(pos); free(req); free(row_idx); free(xd); free(g1d); free(h);
  free(hr); free(pos_r); free(q); free(kv_off); free(prior_off); free(kc); free(vc);
  free(row_n); free(row_ctx); free(row_off); free(o); free(x1); free(g2d); free(h2);
  free(gu); free(a); free(y);
  return 0;
}

/* KV append (vLLM-style paged cache, Section 5.1): a byte copy to the token slots. */
int orc_kv_append(int32_t R, const int32_t* n_new, const int32_t* ctx_len,
                  const int64_t* page_off, const int32_t* pages, int32_t page_size,
                  int32_t nkv, int32_t d, const uint16_t* k_new, const uint16_t* v_new,
                  uint16_t* k_pool, uint16_t* v_pool, int64_t pool_pages) {
  int64_t t = 0;
  for (int32_t r = 0; r < R; r++) {
    for (int32_t i = 0; i < n_new[r]; i++, t++) {
      int64_t p = (int64_t)ctx_len[r] + i;
      int64_t page_index = p / page_size;
      if (page_index >= page_off[r + 1] - page_off[r]) return -1;
      int64_t page = pages[page_off[r] + page_index];
      if (page < 0 || page >= pool_pages) return -1;
      int64_t s = p % page_size;
      for (int32_t g = 0; g < nkv; g++)
        for (int32_t e = 0; e < d; e++) {
          int64_t dst = ((page * nkv + g) * page_size + s) * d + e;
          int64_t src = (t * nkv + g) * d + e;
          k_pool[dst] = k_new[src];
          v_pool[dst] = v_new[src];
        }
    }
  }
  return 0;
}
