// attention.hip -- paged varlen attention for a mixed prefill/decode batch on
// gfx950, one launch over a host-built work list, plus the split merge.
//
// Every wave computes, for up to 16 query rows that share one KV head, the
// transposed score tile S^T = K Q^T (keys x rows) with the 16x16x32 bf16
// matrix-core instruction, and then O^T += V^T P^T.  In that orientation the
// probabilities come out of the first product already in the register layout
// the second product wants as its B operand, and every softmax statistic of a
// query row lives in the lane that also holds that row of O^T, so P never
// leaves registers.  Keys are consumed two pages (32 keys) at a time; the key
// order inside one 32-key step is permuted identically for both products so
// that every key and value load is a 16-byte run.
//
//   decode item : the q heads of one KV-head group of a single decode token,
//                 over one split of the request's pages; the four waves of the
//                 workgroup stride over the split's 32-key chunks and combine
//                 through LDS.  Requests with several splits leave fp32
//                 partials (unnormalised O, running max, running sum) for the
//                 merge kernel.
//   prefill item: one q head, 128 query rows of a prefill chunk (two blocks
//                 of 16 per wave), causal over the cached prefix plus the
//                 chunk; the four waves share each 32-key chunk through LDS
//                 (loaded once per tile), and each wave applies the chunk's
//                 key and value fragments, read from LDS once, to both of its
//                 row blocks.
//
// Masking is select-based: slots at or past the request's length are never
// multiplied into a sum, so stale or NaN-filled slots cannot leak.
#include <type_traits>

#include "mx_device.h"
#include "mx_kernels.h"

namespace mx {

namespace {

constexpr float kNegBig = -1.0e30f;

// Element (token t, column c = head * HD + dim) of the attention output:
// [T][nq][HD] row-major, or the projection-input tile layout when out_tiled.
__device__ __forceinline__ uint16_t* out_ptr(const AttnParams& p, int64_t t, int64_t c) {
  return p.out + (p.out_tiled ? tile_index(t, c, p.out_tok_stride) : t * p.out_tok_stride + c);
}

template <int HD>
struct Chunk {
  u32x4 k[2][HD / 32];  // keys: 16 B per lane per (score block, d-step)
  u32x4 v[HD / 16];     // values (transposed pages): 16 B per lane per d-block
};

// Key order inside a 32-key step (two pages).  Score block b, row m holds key
//   kappa_b(m) = 8 * (m / 4) + 4 * b + m % 4,
// so that lane group g (rows 4g .. 4g+3 of both blocks) ends up with the eight
// consecutive keys 8g .. 8g+7, all in page g / 2.  Those eight keys are then
// one 16-byte run of a transposed value page, and they are exactly the k
// indices the second product expects from this lane group.
// Non-temporal loads (streamed past the caches' retention): every key and
// value of a decode split is read once.  A value load reads whole 128-byte
// lines (16 dim rows x 32 bytes of a page, contiguous), so its values are
// always loaded non-temporally.  Keys are non-temporal (NT) only in launches
// of decode splits alone.  With token-major key pages a key load read half
// lines, and beside prefill tiles (whose copies keep the L2 busy) non-temporal
// keys made the launch slower (70B at P = 4096: 2.19 ms against 1.88 ms); with
// the blocked key pages every key load reads whole lines, and non-temporal
// keys in mixed launches measured no better than ordinary ones.  Measured:
// decode-only attention 3-11% faster on the four layer shapes (7B 70.0 ->
// 78.1% of the HBM peak, 13B 70.6 -> 75.8%, Llama-3-8B 70.8 -> 78.8%, 70B
// 78.2 -> 80.3%); non-temporal values in mixed launches 1-3.5% faster (70B,
// P = 1024 .. 8192).
template <int HD, bool NT>
__device__ __forceinline__ u32x4 stream_load(const uint16_t* ptr) {
  const u32x4* q = reinterpret_cast<const u32x4*>(ptr);
  if constexpr (NT) return __builtin_nontemporal_load(q);
  else return *q;
}

template <int HD, bool NT>
__device__ __forceinline__ void load_chunk(Chunk<HD>& c, const AttnParams& p, int kvh, int pid0,
                                           int pid1, int safe, int col, int g4) {
  // A page id of -1 (past the split's end) reads the request's first page
  // instead: those keys and values are masked out by select in
  // process_chunk, and every load stays unconditional, which keeps the
  // count of loads in flight the same on every path.
  // keys: lane row m = col; its key kappa_b(col) lives in page col / 8.  A key
  // page is blocked by 32 dims ([d / 32][16 slots][32]), so the four
  // consecutive slots that rows 4i .. 4i + 3 read of a 32-dim block in one
  // load are one contiguous 256-byte run: every load moves whole 128-byte
  // lines.
  {
    const int page0 = (col < 8) ? pid0 : pid1;
    const int page = page0 >= 0 ? page0 : safe;
    const int slot0 = 8 * ((col >> 2) & 1) + (col & 3);
    const uint16_t* kb_ptr = p.k_pool + ((int64_t)page * p.nkv + kvh) * (int64_t)(16 * HD);
#pragma unroll
    for (int b = 0; b < 2; b++)
#pragma unroll
      for (int ds = 0; ds < HD / 32; ds++)
        c.k[b][ds] = stream_load<HD, NT>(kb_ptr + ds * 512 + (slot0 + 4 * b) * 32 + 8 * g4);
  }
  // values: lane group g reads keys 8 (g % 2) .. +7 of page g / 2 at d = 16 db + col
  {
    const int page0 = (g4 < 2) ? pid0 : pid1;
    const int page = page0 >= 0 ? page0 : safe;
    const uint16_t* vb_ptr = p.v_pool + ((int64_t)page * p.nkv + kvh) * (int64_t)(16 * HD) + 8 * (g4 & 1);
#pragma unroll
    for (int db = 0; db < HD / 16; db++)
      c.v[db] = stream_load<HD, true>(vb_ptr + (db * 16 + col) * 16);
  }
}

// Online-softmax state of this lane's query row.  m is the running max of the
// scaled scores (log2 units) that every probability of the row refers to, thr
// the raw score above which m has to be raised (m + kLazyMax, unscaled), and
// l this lane's share of the row's sum: the probabilities of the lane's own
// keys only.  The four lanes of a row share m and every rescale, so the row's
// sum is the sum of their shares, taken once at the end.
struct RowState {
  float m, thr, l;
};
__device__ __forceinline__ RowState row_start() { return RowState{kNegBig, kNegBig, 0.f}; }

// A row's running max m (log2 units) is raised only when a score exceeds it by
// more than this: the probabilities exp2(x - m) then stay below 2^8, which bf16
// and fp32 hold at full relative precision, and the output is rescaled only on
// the steps where some row of the wave raised its max (rarely, past the first
// keys).  Output and sum always refer to the same m, so the normalised result
// is the softmax itself.
constexpr float kLazyMax = 8.0f;

// Max and sum of a query row's values over its four lane groups (lanes l,
// l ^ 16, l ^ 32, l ^ 48).  v_permlane16_swap and v_permlane32_swap with both
// operands equal to x leave, in every lane, the even-row (lower-half) value in
// the first result and the odd-row (upper-half) value in the second: the lane's
// own value and its partner's, in the same order in both lanes of a pair.  So
// each step is one VALU swap and one VALU op, with no LDS permute, and the sum
// is bit-identical in the four lanes of a row.
// (The max as compare and select: fmaxf cannot tell that the swapped bits are
// canonical and quiets both operands first, three instructions instead of two.
// Scores are never NaN here: masked keys carry -1e30.)
__device__ __forceinline__ float max_pair(float a, float b) { return a > b ? a : b; }
__device__ __forceinline__ float lane_groups_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = max_pair(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max_pair(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float lane_groups_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// 2^x with the hardware exponential alone (v_exp_f32).  exp2f adds a range
// reduction that keeps results below 2^-126 as denormals (six instructions
// instead of one); a softmax never needs them: every probability is
// 2^(score - m) with the row's running max m at most 2^8 below its largest
// score, so a term under 2^-126 is below 2^-134 of the row's sum and its
// flush to zero changes nothing, and masked scores (-1e30) give exactly 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Score block b of S^T = K Q^T (16 keys x 16 rows).
template <int HD>
__device__ __forceinline__ f32x4 score_block(const u32x4 (&kf)[HD / 32], const bf16x8 (&qf)[HD / 32]) {
  f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ds = 0; ds < HD / 32; ds++) s = mfma16(as_bf16x8(kf[ds]), qf[ds], s);
  return s;
}

// This lane's eight raw scores of the step (keys past the range or after the
// row's position masked to kNegBig by select) and their max.
template <bool MASK>
__device__ __forceinline__ float masked_scores(const f32x4 (&s)[2], float (&sv)[2][4], int pi0,
                                               int page_end, int row_pos, int g4) {
  const bool pvalid = (pi0 + (g4 >> 1)) < page_end;
  const int j0 = pi0 * 16 + 8 * g4;
  float mx = kNegBig;
#pragma unroll
  for (int b = 0; b < 2; b++)
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int j = j0 + 4 * b + i;
      sv[b][i] = (!MASK || (pvalid && j <= row_pos)) ? s[b][i] : kNegBig;
      mx = fmaxf(mx, sv[b][i]);
    }
  return mx;
}

// Called by the whole wave when some lane holds a score above its row's
// threshold: each row takes its max over its four lane groups and raises m to
// it if that exceeds m by more than kLazyMax, rescaling its output and sum.
// The first step of every row comes here (thr starts at kNegBig and every row
// has a key in its first step).
template <int NO>
__device__ __forceinline__ void raise_max(RowState& r, float mx, float scale_log2, float inv_scale,
                                          f32x4 (&o)[NO]) {
  const float rmx = lane_groups_max(mx) * scale_log2;  // scale > 0: the max of the scaled scores
  const bool raise = rmx > r.m + kLazyMax;
  const float m_new = raise ? rmx : r.m;
  const float alpha = raise ? fast_exp2(r.m - m_new) : 1.f;
#pragma unroll
  for (int e = 0; e < NO; e++) o[e] = o[e] * alpha;
  r.l *= alpha;
  r.m = m_new;
  r.thr = (m_new + kLazyMax) * inv_scale;
}

// The step's probabilities of this lane's keys, exp2(score * scale - m), as
// the value product's B operand (k index i' = 4 b + i <-> key j0 + i'), and
// their sum into the lane's share of the row's sum: two at a time with the
// bf16 dot instruction, from the same rounded values the value product uses.
__device__ __forceinline__ bf16x8 probs(const float (&sv)[2][4], RowState& r, float scale_log2) {
  float pv[2][4];
#pragma unroll
  for (int b = 0; b < 2; b++)
#pragma unroll
    for (int i = 0; i < 4; i++) pv[b][i] = fast_exp2(fmaf(sv[b][i], scale_log2, -r.m));
  // Four separate words, put together only for the return: with the words
  // taken out of a four-word vector, this compiler's dot instructions all
  // read its first word.
  const uint32_t w0 = pack_bf16x2(pv[0][0], pv[0][1]);
  const uint32_t w1 = pack_bf16x2(pv[0][2], pv[0][3]);
  const uint32_t w2 = pack_bf16x2(pv[1][0], pv[1][1]);
  const uint32_t w3 = pack_bf16x2(pv[1][2], pv[1][3]);
  const mx_bf16x2 ones = __builtin_bit_cast(mx_bf16x2, 0x3F803F80u);
  r.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(mx_bf16x2, w0), ones, r.l, false);
  r.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(mx_bf16x2, w1), ones, r.l, false);
  r.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(mx_bf16x2, w2), ones, r.l, false);
  r.l = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(mx_bf16x2, w3), ones, r.l, false);
  return as_bf16x8(u32x4{w0, w1, w2, w3});
}

// Which of this lane group's eight keys hold values (bf16 lanes of each
// 32-bit word): keys past the request's length are zeroed by select, not
// multiplied, so that NaN-filled slots stay out of the sum.  Depends on the
// keys only, not on the row.
__device__ __forceinline__ void value_keep(int pi0, int page_end, int kv_len, int g4,
                                           uint32_t (&keep)[4]) {
  const bool pvalid = (pi0 + (g4 >> 1)) < page_end;
  const int j0 = pi0 * 16 + 8 * g4;
#pragma unroll
  for (int h = 0; h < 4; h++) {
    const bool k0 = pvalid && (j0 + 2 * h) < kv_len;
    const bool k1 = pvalid && (j0 + 2 * h + 1) < kv_len;
    keep[h] = (k0 ? 0x0000FFFFu : 0u) | (k1 ? 0xFFFF0000u : 0u);
  }
}

// O^T += V^T P^T over the output blocks DB0 .. DB0 + NDB - 1 (16 head dims
// each), V^T as the A operand.
template <int HD, int DB0, int NDB, bool MASK>
__device__ __forceinline__ void values_part(const u32x4 (&vf)[NDB], f32x4 (&o)[HD / 16], bf16x8 pb,
                                            const uint32_t (&keep)[4]) {
#pragma unroll
  for (int e = 0; e < NDB; e++) {
    u32x4 va = vf[e];
    if constexpr (MASK) {
#pragma unroll
      for (int h = 0; h < 4; h++) va[h] &= keep[h];
    }
    o[DB0 + e] = mfma16(as_bf16x8(va), pb, o[DB0 + e]);
  }
}

// One 32-key step of the online softmax for this lane's query row.  Lane group
// g4 owns keys pi0 * 16 + 8 * g4 + i' (i' = 4 b + i for score block b, row i).
template <int HD, bool MASK = true>
__device__ __forceinline__ void process_chunk(const Chunk<HD>& c, const bf16x8 (&qf)[HD / 32],
                                              f32x4 (&o)[HD / 16], RowState& r, int pi0,
                                              int page_end, int row_pos, int kv_len,
                                              float scale_log2, float inv_scale, int g4) {
  const f32x4 s[2] = {score_block<HD>(c.k[0], qf), score_block<HD>(c.k[1], qf)};
  float sv[2][4];
  const float mx = masked_scores<MASK>(s, sv, pi0, page_end, row_pos, g4);
  if (__any(mx > r.thr)) raise_max(r, mx, scale_log2, inv_scale, o);
  const bf16x8 pb = probs(sv, r, scale_log2);
  uint32_t keep[4];
  value_keep(pi0, page_end, kv_len, g4, keep);
  values_part<HD, 0, HD / 16, MASK>(c.v, o, pb, keep);
}

// Keys pi0 * 16 .. pi0 * 16 + 31 all count for every row of the wave (both
// pages inside the range, and the chunk's last key at or before the wave's
// first row position, which is below kv_len): no mask is needed.
__device__ __forceinline__ bool chunk_interior(int pi0, int page_end, int first_row_pos) {
  return pi0 + 1 < page_end && pi0 * 16 + 31 <= first_row_pos;
}

// Prefill tiles share every 32-key chunk through LDS.  The four waves copy it
// there with the DMA path (global_load_lds, 16 bytes per lane), a quarter each
// (waves 0 and 1 the keys of the chunk's two pages, waves 2 and 3 their
// values), and every wave reads its matrix-core fragments from there.  Keys
// are stored [32][HD] with the 16-byte chunk c of key row j at c ^ ksw(j);
// values page by page, [2 pages][HD][2 halves of 8 keys], with half h of dim
// row d at h ^ ((d >> 3) & 1).  Both make the fragment reads (16 key rows, or
// 16 dim rows, at one logical chunk) hit distinct bank groups.  A DMA
// instruction writes 1 KB of LDS in lane order, so each lane fetches the 16
// bytes that belong at its position: a permutation within the page's rows
// (and, for keys, within its 32-dim blocks), which keeps every copy a run of
// whole 128-byte lines.  Each copy instruction reads from one page only, so
// its page address is the same for every lane (scalar arithmetic; with the
// values' two pages side by side in every dim row, as first laid out, the
// lanes of one copy read from both, and choosing and forming a 64-bit address
// per lane cost 14 of the loop's 81 vector instructions per chunk).
template <int HD>
__device__ __forceinline__ int ksw(int key) {
  if constexpr (HD == 128) return (key & 3) | ((key >> 3) << 2);
  else return ((key >> 1) & 1) | ((key >> 3) << 1);
}
template <int HD>
struct SharedChunk {
  static constexpr int KBYTES = 32 * HD * 2;
  static constexpr int BYTES = 2 * KBYTES;  // keys + values
  static constexpr int SLOTS = 4;           // chunks kt .. kt + 3: copies run three ahead
  static constexpr int NLD = BYTES / 4096;  // 1 KB copies per wave per chunk
};
template <int HD>
constexpr int smem_bytes() {
  constexpr int ring = SharedChunk<HD>::SLOTS * SharedChunk<HD>::BYTES;
  constexpr int combine = (4 * 16 * (HD + 4) + 2 * 4 * 16) * 4;
  return ring > combine ? ring : combine;
}

// v[e] = the 16 bytes at LDS address addr + OFF0 + e * STEP, e = E .. N - 1.
template <int E, int N, int OFF0, int STEP>
__device__ __forceinline__ void lds_read_run(unsigned addr, u32x4 (&v)[N]) {
  if constexpr (E < N) {
    v[E] = lds_read16_at<OFF0 + E * STEP>(addr);
    lds_read_run<E + 1, N, OFF0, STEP>(addr, v);
  }
}

// Prefill item: one q head, rows it.start .. it.start + 127 of the chunk; wave
// w owns two blocks of 16 consecutive rows, it.start + 32 w + (0 | 16) + col.
//
// Iteration kt of the chunk loop reads the keys of chunk kt + 1 for the score
// products while the exponentials of chunk kt (whose scores the previous
// iteration left) run on the vector units, then takes the value products of
// chunk kt, and raises the rows' running max for chunk kt + 1 where needed:
// the scores of the next chunk and the softmax of the current one are
// independent, so they share a basic block and the matrix cores have work
// while the exponentials run.  The copies of chunk kt + 3 go out at the top of
// iteration kt into the slot chunk kt - 1 used, after the barrier that ends
// every wave's reads of it; page ids are loaded one iteration before their
// copies.  Every iteration issues the same copies (chunks past the tile's last
// one copy the request's first page into the free slot and are never read),
// and they are the only vector-memory operations of the loop (page ids are
// scalar loads), so one vmcnt value fits every wait: at the top of iteration
// kt the copies of iteration kt - 1 may still be in flight, every earlier one
// (chunk kt + 1) has landed.
static_assert(kPrefillTileRows == 4 * 32, "four waves of two 16-row blocks");
template <int HD>
__device__ __forceinline__ void prefill_item(const AttnParams& p, const AttnItem& it,
                                             const ReqDev& rq, char* smem) {
  using SC = SharedChunk<HD>;
  constexpr int KB = SC::KBYTES, CB = SC::BYTES, NLD = SC::NLD, ND = HD / 32;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15;  // query row of this lane within each block
  const int g4 = lane >> 4;   // lane group
  const int qhead = it.head;
  const int kvh = qhead / p.group;
  const int row0 = it.start + 32 * wave;
  const int row = row0 + col, row2 = row0 + 16 + col;
  const bool row_valid = row < rq.n_new, row_valid2 = row2 < rq.n_new;
  const int rowc = row_valid ? row : rq.n_new - 1;
  const int rowc2 = row_valid2 ? row2 : rq.n_new - 1;
  const int64_t qtok = rq.tok_start + rowc, qtok2 = rq.tok_start + rowc2;
  const int row_pos = rq.ctx_len + rowc, row_pos2 = rq.ctx_len + rowc2;
  const int last_row = min(row0 + 31, rq.n_new - 1);
  const int page_end = row0 < rq.n_new ? (rq.ctx_len + last_row) / 16 + 1 : 0;

  bf16x8 qf[ND], qf2[ND];
  {
    const uint16_t* qp = p.q + qtok * p.q_tok_stride + (int64_t)qhead * HD + 8 * g4;
    const uint16_t* qp2 = p.q + qtok2 * p.q_tok_stride + (int64_t)qhead * HD + 8 * g4;
#pragma unroll
    for (int ds = 0; ds < ND; ds++) {
      u32x4 v = row_valid ? *reinterpret_cast<const u32x4*>(qp + ds * 32) : u32x4{0, 0, 0, 0};
      u32x4 v2 = row_valid2 ? *reinterpret_cast<const u32x4*>(qp2 + ds * 32) : u32x4{0, 0, 0, 0};
      qf[ds] = as_bf16x8(v);
      qf2[ds] = as_bf16x8(v2);
    }
  }
  RowState r1 = row_start(), r2 = row_start();
  const float inv_scale = 1.f / p.scale_log2;
  f32x4 o[HD / 16], o2[HD / 16];
#pragma unroll
  for (int db = 0; db < HD / 16; db++) o[db] = o2[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  // the tile's last row bounds the pages every wave helps to copy
  const int tile_last = min(it.start + kPrefillTileRows - 1, rq.n_new - 1);
  const int item_pages = (rq.ctx_len + tile_last) / 16 + 1;
  const int n_chunks = (item_pages + 1) / 2;
  const int wave_chunks = (page_end + 1) / 2;  // 0 for a wave without valid rows
  const int wave_first_pos = rq.ctx_len + it.start + 32 * wave;  // the wave's first row
  // page ids through the constant address space: uniform reads of a table
  // nothing writes during the launch, so they are scalar loads, whose
  // results the compiler waits for with lgkmcnt when it uses them (vector
  // loads would put the compiler's own vmcnt waits among the copies)
  const __attribute__((address_space(4))) int32_t* ptab =
      (const __attribute__((address_space(4))) int32_t*)(p.pages + rq.page_start);
  const int last_page = rq.n_pages - 1;
  const int safe = ptab[0];

  // This lane's share of the wave's 1 KB copies: copy i fills LDS kilobyte
  // kb = NLD * wave + i of the slot (keys first, then values) with the 16 bytes
  // at element offset off[i] of the chunk's first (sel[i] false) or second page.
  int off[NLD];
  bool sel[NLD];  // (the same for every lane: each copy reads one page)
#pragma unroll
  for (int i = 0; i < NLD; i++) {
    const int kb = NLD * wave + i;
    if (wave < 2) {
      constexpr int lanes_per_row = HD / 8;  // 16-byte pieces of a key row
      const int j = kb * (64 / lanes_per_row) + lane / lanes_per_row;
      const int lc = (lane % lanes_per_row) ^ ksw<HD>(j);
      sel[i] = kb * (64 / lanes_per_row) >= 16;
      off[i] = (lc >> 2) * 512 + (j & 15) * 32 + (lc & 3) * 8;
    } else {
      // values: [page][dim][2 halves of 8 keys], half h of dim row d stored
      // at h ^ ((d >> 3) & 1)
      const int vb = (kb - KB / 1024) * 1024 + lane * 16;  // byte in the value half
      const int d = (vb % (HD * 32)) / 32;
      const int h = ((vb / 16) & 1) ^ ((d >> 3) & 1);
      sel[i] = (kb - KB / 1024) * 1024 >= HD * 32;
      off[i] = d * 16 + h * 8;
    }
  }
  const uint16_t* pool = wave < 2 ? p.k_pool : p.v_pool;
  const unsigned lds0 = (unsigned)(size_t)(MX_LDS char*)smem;
  auto copy = [&](int c, int ra, int rb) {  // ra, rb: page ids of pages 2c, 2c + 1
    const int pa = 2 * c < item_pages ? ra : safe;
    const int pb = 2 * c + 1 < item_pages ? rb : safe;
    const uint16_t* ba = pool + ((int64_t)pa * p.nkv + kvh) * (16 * HD);
    const uint16_t* bb = pool + ((int64_t)pb * p.nkv + kvh) * (16 * HD);
    const unsigned dst = lds0 + (unsigned)((c & 3) * CB + NLD * wave * 1024);
#pragma unroll
    for (int i = 0; i < NLD; i++) {
      dma16((sel[i] ? bb : ba) + off[i], dst + i * 1024);
    }
  };
  auto page_of = [&](int pi) { return ptab[min(pi, last_page)]; };

  // fragment addresses within a slot: key rows kappa_0(col) (score block 1 is
  // four key rows further, same swizzle), value dim rows 16 e + col
  const int key0 = 16 * (col >> 3) + 8 * ((col >> 2) & 1) + (col & 3);
  unsigned kaddr[ND];
#pragma unroll
  for (int ds = 0; ds < ND; ds++)
    kaddr[ds] = (unsigned)(key0 * (HD * 2) + (((4 * ds + g4) ^ ksw<HD>(key0)) << 4));
  const unsigned vaddr = (unsigned)(KB + (g4 >> 1) * (HD * 32) + col * 32 +
                                    (((g4 & 1) ^ ((col >> 3) & 1)) << 4));

  // scores of chunk c from its keys in LDS: this lane's masked raw scores, their
  // max, and whether some lane of the wave is above its row's threshold
  float sv1[2][4], sv2[2][4], mx1 = kNegBig, mx2 = kNegBig;
  auto scores = [&](auto mask, int c) -> bool {
    constexpr bool MASK = decltype(mask)::value;
    const unsigned sb = lds0 + (unsigned)((c & 3) * CB);
    u32x4 k0[ND], k1[ND];
#pragma unroll
    for (int ds = 0; ds < ND; ds++) k0[ds] = lds_read16(sb + kaddr[ds]);
#pragma unroll
    for (int ds = 0; ds < ND; ds++) k1[ds] = lds_read16_at<4 * HD * 2>(sb + kaddr[ds]);
    f32x4 s1[2], s2[2];
    lgkm_wait<ND>();
    pin(k0);
    s1[0] = score_block<HD>(k0, qf);
    s2[0] = score_block<HD>(k0, qf2);
    __builtin_amdgcn_sched_barrier(0);  // these products go before the second wait
    lgkm_wait<0>();
    pin(k1);
    s1[1] = score_block<HD>(k1, qf);
    s2[1] = score_block<HD>(k1, qf2);
    mx1 = masked_scores<MASK>(s1, sv1, 2 * c, page_end, row_pos, g4);
    mx2 = masked_scores<MASK>(s2, sv2, 2 * c, page_end, row_pos2, g4);
    return __any(mx1 > r1.thr || mx2 > r2.thr) != 0;
  };
  // value products of chunk c (values past the request's keys zeroed when
  // MASK: only the chunk that holds the request's last key has such values)
  auto values = [&](auto mask, int c, bf16x8 pb1, bf16x8 pb2) {
    constexpr bool MASK = decltype(mask)::value;
    const unsigned va = lds0 + (unsigned)((c & 3) * CB) + vaddr;
    u32x4 v0[ND], v1[ND];
    lds_read_run<0, ND, 0, 512>(va, v0);
    lds_read_run<0, ND, ND * 512, 512>(va, v1);
    uint32_t keep[4] = {~0u, ~0u, ~0u, ~0u};
    if constexpr (MASK) value_keep(2 * c, page_end, rq.kv_len, g4, keep);
    lgkm_wait<ND>();
    pin(v0);
    values_part<HD, 0, ND, MASK>(v0, o, pb1, keep);
    values_part<HD, 0, ND, MASK>(v0, o2, pb2, keep);
    __builtin_amdgcn_sched_barrier(0);  // these products go before the second wait
    lgkm_wait<0>();
    pin(v1);
    values_part<HD, ND, ND, MASK>(v1, o, pb1, keep);
    values_part<HD, ND, ND, MASK>(v1, o2, pb2, keep);
  };
  auto raise_rows = [&]() {
    raise_max(r1, mx1, p.scale_log2, inv_scale, o);
    raise_max(r2, mx2, p.scale_log2, inv_scale, o2);
  };
  using Masked = std::integral_constant<bool, true>;
  using Unmasked = std::integral_constant<bool, false>;

  // prologue: page ids of chunks 0 .. 3, the copies of chunks 0 .. 2
  int ua, ub, fa = 0, fb = 0;  // page ids of the chunk the next copy is for, and the one after
  {
    const int a0 = page_of(0), b0 = page_of(1), a1 = page_of(2), b1 = page_of(3);
    const int a2 = page_of(4), b2 = page_of(5);
    copy(0, a0, b0);
    copy(1, a1, b1);
    ua = page_of(6);
    ub = page_of(7);
    copy(2, a2, b2);
  }
  // top of iteration kt: this wave's copies of chunk kt + 1 have landed, then
  // everyone's, and every read of chunk kt - 1 is done; chunk kt + 3 goes out
  auto top = [&](int kt, int& use_a, int& use_b, int& fill_a, int& fill_b) {
    vm_wait<NLD>();
    wg_barrier();
    fill_a = page_of(2 * (kt + 4));
    fill_b = page_of(2 * (kt + 4) + 1);
    copy(kt + 3, use_a, use_b);
  };
  auto run = [&](int kt0, int kt1, auto body) {  // iterations kt0 .. kt1 - 1
    for (int kt = kt0; kt < kt1; kt += 2) {
      top(kt, ua, ub, fa, fb);
      body(kt);
      if (kt + 1 >= kt1) {  // an odd count: the next iteration uses fa, fb
        const int ta = ua, tb = ub;
        ua = fa;
        ub = fb;
        fa = ta;
        fb = tb;
        break;
      }
      top(kt + 1, fa, fb, ua, ub);
      body(kt + 1);
    }
  };

  if (row0 >= rq.n_new) {
    // no rows here: this wave only copies its quarter of every chunk
    vm_wait<2 * NLD>();
    wg_barrier();
    run(0, n_chunks, [](int) {});
    vm_wait<0>();  // no copy may land in LDS after the workgroup has ended
    return;
  }

  vm_wait<2 * NLD>();  // chunk 0 has landed; chunks 1 and 2 may be in flight
  wg_barrier();
  if (scores(Masked{}, 0)) raise_rows();  // the first step raises every row's max

  // Chunks 0 .. n_int - 1 are inside every wave's range and at or before
  // every row of the tile: no masks.  The last chunk of the tile is the only
  // one that can hold keys past the request's end, so n_main <= n_chunks - 1.
  const int first_pos = rq.ctx_len + it.start;
  const int page_end0 = (rq.ctx_len + min(it.start + 31, rq.n_new - 1)) / 16 + 1;  // wave 0's
  const int n_int = first_pos >= 31 ? min((first_pos - 31) / 32 + 1, page_end0 / 2) : 0;
  const int n_main = max(0, n_int - 1);
  // main loop: the scores of chunk kt + 1 and the softmax of chunk kt in one
  // basic block, then the values of chunk kt; no masks, no per-wave bounds
  run(0, n_main, [&](int kt) {
    const bf16x8 pb1 = probs(sv1, r1, p.scale_log2);
    const bf16x8 pb2 = probs(sv2, r2, p.scale_log2);
    const bool raise = scores(Unmasked{}, kt + 1);
    values(Unmasked{}, kt, pb1, pb2);
    if (raise) raise_rows();
  });
  // the chunks around the diagonal and the tile's end, with masks and bounds
  run(n_main, n_chunks, [&](int kt) {
    const bool sc = kt + 1 < wave_chunks;  // scores of chunk kt + 1
    if (kt < wave_chunks) {
      const bf16x8 pb1 = probs(sv1, r1, p.scale_log2);
      const bf16x8 pb2 = probs(sv2, r2, p.scale_log2);
      values(Masked{}, kt, pb1, pb2);
    }
    if (sc && scores(Masked{}, kt + 1)) raise_rows();
  });
  vm_wait<0>();  // no copy may land in LDS after the workgroup has ended

  // the rows' sums over their four lane groups (every lane takes part)
  const float l1 = lane_groups_sum(r1.l), l2 = lane_groups_sum(r2.l);
  // dims 16 db + 4 g4 .. + 3 of the row: (db / 2) 32-column steps plus 16 (db % 2)
  const int64_t step32 = p.out_tiled ? 512 : 32;
  if (row_valid) {
    const float inv = 1.f / l1;
    uint16_t* op = out_ptr(p, qtok, qhead * HD + 4 * g4);
#pragma unroll
    for (int db = 0; db < HD / 16; db++) {
      u32x2 w;
      w[0] = pack_bf16x2(o[db][0] * inv, o[db][1] * inv);
      w[1] = pack_bf16x2(o[db][2] * inv, o[db][3] * inv);
      *reinterpret_cast<u32x2*>(op + (db >> 1) * step32 + (db & 1) * 16) = w;
    }
  }
  if (row_valid2) {
    const float inv = 1.f / l2;
    uint16_t* op = out_ptr(p, qtok2, qhead * HD + 4 * g4);
#pragma unroll
    for (int db = 0; db < HD / 16; db++) {
      u32x2 w;
      w[0] = pack_bf16x2(o2[db][0] * inv, o2[db][1] * inv);
      w[1] = pack_bf16x2(o2[db][2] * inv, o2[db][3] * inv);
      *reinterpret_cast<u32x2*>(op + (db >> 1) * step32 + (db & 1) * 16) = w;
    }
  }
}

// Decode item: the q heads it.head .. it.head + nrows - 1 (one per lane row)
// of the request's single token, over pages it.start .. of its table; the four
// waves stride over the split's 32-key chunks and combine through LDS.
template <int HD, bool NT>
__device__ __forceinline__ void decode_item(const AttnParams& p, const AttnItem& it,
                                            const ReqDev& rq, char* smem) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;  // q head of this lane (relative to it.head)
  const int g4 = lane >> 4;   // lane group
  const int qhead = it.head + col;
  const bool row_valid = col < it.nrows;
  const int kvh = it.head / p.group;
  const int64_t qtok = rq.tok_start;
  const int row_pos = rq.kv_len - 1;
  const int page_end = min(it.start + p.split_pages, rq.n_pages);
  const int chunk_first = it.start + 2 * wave;
  constexpr int chunk_step = 8;

  RowState r = row_start();
  const float inv_scale = 1.f / p.scale_log2;
  f32x4 o[HD / 16];
#pragma unroll
  for (int db = 0; db < HD / 16; db++) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 qf[HD / 32];
  {
    const uint16_t* qp = p.q + qtok * p.q_tok_stride + (int64_t)qhead * HD + 8 * g4;
#pragma unroll
    for (int ds = 0; ds < HD / 32; ds++) {
      u32x4 v = row_valid ? *reinterpret_cast<const u32x4*>(qp + ds * 32) : u32x4{0, 0, 0, 0};
      qf[ds] = as_bf16x8(v);
    }
  }

  // Two chunk buffers used in turn: the loads of the next chunk are in flight
  // while the current one is processed.  The loop is unrolled by two so that
  // no buffer is ever copied (a register copy of a buffer whose loads are in
  // flight waits for them and serialises the prefetch), and a chunk's loads
  // are issued only on the path where that chunk exists, unconditionally
  // there, so the compiler's wait before each chunk covers exactly its own
  // loads.  Page ids are fetched one chunk ahead of their loads.
  const int safe = p.pages[rq.page_start];
  auto pid = [&](int pi) -> int {
    const int v = p.pages[rq.page_start + min(pi, rq.n_pages - 1)];
    return pi < page_end ? v : -1;
  };
  auto proc = [&](const Chunk<HD>& c, int pi0) {
    if (chunk_interior(pi0, page_end, row_pos))
      process_chunk<HD, false>(c, qf, o, r, pi0, page_end, row_pos, rq.kv_len, p.scale_log2,
                               inv_scale, g4);
    else
      process_chunk<HD>(c, qf, o, r, pi0, page_end, row_pos, rq.kv_len, p.scale_log2, inv_scale,
                        g4);
  };
  Chunk<HD> ca, cb;
  int pi = chunk_first;
  if (pi < page_end) {
    int n0 = pid(pi + chunk_step), n1 = pid(pi + chunk_step + 1);
    load_chunk<HD, NT>(ca, p, kvh, pid(pi), pid(pi + 1), safe, col, g4);
    while (true) {
      int pn = pi + chunk_step;
      if (pn >= page_end) {
        proc(ca, pi);
        break;
      }
      int nn0 = pid(pn + chunk_step), nn1 = pid(pn + chunk_step + 1);
      load_chunk<HD, NT>(cb, p, kvh, n0, n1, safe, col, g4);
      proc(ca, pi);
      pi = pn;
      n0 = nn0;
      n1 = nn1;
      pn = pi + chunk_step;
      if (pn >= page_end) {
        proc(cb, pi);
        break;
      }
      nn0 = pid(pn + chunk_step);
      nn1 = pid(pn + chunk_step + 1);
      load_chunk<HD, NT>(ca, p, kvh, n0, n1, safe, col, g4);
      proc(cb, pi);
      pi = pn;
      n0 = nn0;
      n1 = nn1;
    }
  }

  // decode: combine the four waves' partial softmax states through LDS
  float(*s_o)[16][HD + 4] = reinterpret_cast<float(*)[16][HD + 4]>(smem);
  float(*s_m)[16] = reinterpret_cast<float(*)[16]>(smem + 4 * 16 * (HD + 4) * 4);
  float(*s_l)[16] = reinterpret_cast<float(*)[16]>(smem + 4 * 16 * (HD + 4) * 4 + 4 * 16 * 4);
#pragma unroll
  for (int db = 0; db < HD / 16; db++)
#pragma unroll
    for (int i = 0; i < 4; i++) s_o[wave][col][db * 16 + 4 * g4 + i] = o[db][i];
  const float l = lane_groups_sum(r.l);
  if (g4 == 0) {
    s_m[wave][col] = r.m;
    s_l[wave][col] = l;
  }
  __syncthreads();
  const int row = threadIdx.x >> 4;         // 16 rows
  const int dseg = (threadIdx.x & 15) * (HD / 16);
  if (row >= it.nrows) return;
  float M = kNegBig;
#pragma unroll
  for (int w = 0; w < 4; w++) M = fmaxf(M, s_m[w][row]);
  float wt[4], L = 0.f;
#pragma unroll
  for (int w = 0; w < 4; w++) {
    wt[w] = exp2f(s_m[w][row] - M);
    L += s_l[w][row] * wt[w];
  }
  float acc[HD / 16];
#pragma unroll
  for (int e = 0; e < HD / 16; e++) {
    float a = 0.f;
#pragma unroll
    for (int w = 0; w < 4; w++) a += s_o[w][row][dseg + e] * wt[w];
    acc[e] = a;
  }
  const int h = it.head + row;
  if (rq.n_split == 1) {
    const float inv = 1.f / L;
    uint16_t* op = out_ptr(p, qtok, h * HD + dseg);  // HD / 16 dims within a 32-column block
#pragma unroll
    for (int e = 0; e < HD / 16; e += 2)
      *reinterpret_cast<uint32_t*>(op + e) = pack_bf16x2(acc[e] * inv, acc[e + 1] * inv);
  } else {
    const int64_t part = (int64_t)it.part + (int64_t)row * rq.n_split;
    float* po = p.part_o + part * HD + dseg;
#pragma unroll
    for (int e = 0; e < HD / 16; e += 4)
      *reinterpret_cast<f32x4*>(po + e) = f32x4{acc[e], acc[e + 1], acc[e + 2], acc[e + 3]};
    if ((threadIdx.x & 15) == 0) {
      p.part_ml[part * 2 + 0] = M;
      p.part_ml[part * 2 + 1] = L;
    }
  }
}

template <int HD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void paged_attn_kernel(AttnParams p) {
  __shared__ __attribute__((aligned(16))) char smem[smem_bytes<HD>()];
  const AttnItem it = p.items[blockIdx.x];
  const ReqDev rq = p.reqs[it.req];
  if (it.kind == 1)
    prefill_item<HD>(p, it, rq, smem);
  else if (p.decode_only)
    decode_item<HD, true>(p, it, rq, smem);
  else
    decode_item<HD, false>(p, it, rq, smem);
}

// Deterministic merge of the key splits of one (decode request, q head).
template <int HD>
__global__ __launch_bounds__(HD) void attn_merge_kernel(AttnParams p, const MergeItem* merges) {
  const MergeItem mi = merges[blockIdx.x];
  const ReqDev rq = p.reqs[mi.req];
  const int h = blockIdx.y;
  const int d = threadIdx.x;
  const int ns = rq.n_split;
  const int64_t base = (int64_t)mi.part_base + (int64_t)h * ns;
  float M = kNegBig;
  for (int s = 0; s < ns; s++) M = fmaxf(M, p.part_ml[(base + s) * 2]);
  float L = 0.f, acc = 0.f;
  for (int s = 0; s < ns; s++) {
    const float w = exp2f(p.part_ml[(base + s) * 2] - M);
    L += p.part_ml[(base + s) * 2 + 1] * w;
    acc += p.part_o[(base + s) * HD + d] * w;
  }
  *out_ptr(p, rq.tok_start, h * HD + d) = f32_to_bf16(acc / L);
}

}  // namespace

hipError_t launch_paged_attn(const AttnParams& p, int n_items, const MergeItem* merges,
                             int n_merges, int head_dim, hipStream_t stream) {
  if (n_items > 0) {
    if (head_dim == 128)
      paged_attn_kernel<128><<<n_items, 256, 0, stream>>>(p);
    else
      paged_attn_kernel<64><<<n_items, 256, 0, stream>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (n_merges > 0) {
    dim3 grid(n_merges, p.nq);
    if (head_dim == 128)
      attn_merge_kernel<128><<<grid, 128, 0, stream>>>(p, merges);
    else
      attn_merge_kernel<64><<<grid, 64, 0, stream>>>(p, merges);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace mx
