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
template <int HD>
__device__ __forceinline__ void load_chunk(Chunk<HD>& c, const AttnParams& p, int kvh, int pid0,
                                           int pid1, int safe, int col, int g4) {
  // A page id of -1 (past the split's end) reads the request's first page
  // instead: those keys and values are masked out by select in
  // process_chunk, and every load stays unconditional, which keeps the
  // count of loads in flight the same on every path.
  // keys: lane row m = col; its key kappa_b(col) lives in page col / 8
  {
    const int page0 = (col < 8) ? pid0 : pid1;
    const int page = page0 >= 0 ? page0 : safe;
    const int slot0 = 8 * ((col >> 2) & 1) + (col & 3);
    const uint16_t* kb_ptr = p.k_pool + ((int64_t)page * p.nkv + kvh) * (int64_t)(16 * HD);
#pragma unroll
    for (int b = 0; b < 2; b++)
#pragma unroll
      for (int ds = 0; ds < HD / 32; ds++)
        c.k[b][ds] = *reinterpret_cast<const u32x4*>(kb_ptr + (slot0 + 4 * b) * HD + ds * 32 + 8 * g4);
  }
  // values: lane group g reads keys 8 (g % 2) .. +7 of page g / 2 at d = 16 db + col
  {
    const int page0 = (g4 < 2) ? pid0 : pid1;
    const int page = page0 >= 0 ? page0 : safe;
    const uint16_t* vb_ptr = p.v_pool + ((int64_t)page * p.nkv + kvh) * (int64_t)(16 * HD) + 8 * (g4 & 1);
#pragma unroll
    for (int db = 0; db < HD / 16; db++)
      c.v[db] = *reinterpret_cast<const u32x4*>(vb_ptr + (db * 16 + col) * 16);
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

// Prefill tiles share every 32-key chunk through LDS: the four waves load it
// once, a quarter each (waves 0 and 1 the keys of the chunk's two pages, waves
// 2 and 3 their values), and every wave reads its matrix-core fragments from
// there.  Keys are stored [32][HD] with the 16-byte chunk c of key row j at
// c ^ ksw(j); values [HD][32 keys] with the 16-byte chunk c of dim row d at
// c ^ ((d >> 2) & 3).  Both make the fragment reads (16 key rows, or 16 dim
// rows, at one logical chunk) and the stores hit distinct bank groups.
template <int HD>
__device__ __forceinline__ int ksw(int key) {
  if constexpr (HD == 128) return (key & 3) | ((key >> 3) << 2);
  else return ((key >> 1) & 1) | ((key >> 3) << 1);
}
template <int HD>
struct SharedChunk {
  static constexpr int KBYTES = 32 * HD * 2;
  static constexpr int BYTES = 2 * KBYTES;  // keys + values
};
template <int HD>
constexpr int smem_bytes() {
  constexpr int ring = 2 * SharedChunk<HD>::BYTES;
  constexpr int combine = (4 * 16 * (HD + 4) + 2 * 4 * 16) * 4;
  return ring > combine ? ring : combine;
}

// Prefill item: one q head, rows it.start .. it.start + 127 of the chunk; wave
// w owns two blocks of 16 consecutive rows, it.start + 32 w + (0 | 16) + col.
static_assert(kPrefillTileRows == 4 * 32, "four waves of two 16-row blocks");
template <int HD>
__device__ __forceinline__ void prefill_item(const AttnParams& p, const AttnItem& it,
                                             const ReqDev& rq, char* smem) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
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

  RowState r1 = row_start(), r2 = row_start();
  const float inv_scale = 1.f / p.scale_log2;
  f32x4 o[HD / 16], o2[HD / 16];
#pragma unroll
  for (int db = 0; db < HD / 16; db++) o[db] = o2[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 qf[HD / 32], qf2[HD / 32];
  {
    const uint16_t* qp = p.q + qtok * p.q_tok_stride + (int64_t)qhead * HD + 8 * g4;
    const uint16_t* qp2 = p.q + qtok2 * p.q_tok_stride + (int64_t)qhead * HD + 8 * g4;
#pragma unroll
    for (int ds = 0; ds < HD / 32; ds++) {
      u32x4 v = row_valid ? *reinterpret_cast<const u32x4*>(qp + ds * 32) : u32x4{0, 0, 0, 0};
      u32x4 v2 = row_valid2 ? *reinterpret_cast<const u32x4*>(qp2 + ds * 32) : u32x4{0, 0, 0, 0};
      qf[ds] = as_bf16x8(v);
      qf2[ds] = as_bf16x8(v2);
    }
  }

  // the tile's last row bounds the pages every wave helps to load
  const int tile_last = min(it.start + kPrefillTileRows - 1, rq.n_new - 1);
  const int item_pages = (rq.ctx_len + tile_last) / 16 + 1;
  const int n_chunks = (item_pages + 1) / 2;
  const int wave_chunks = (page_end + 1) / 2;  // 0 for a wave without valid rows
  const int wave_first_pos = rq.ctx_len + it.start + 32 * wave;  // the wave's first row
  const int safe = p.pages[rq.page_start];
  auto pid = [&](int pi) -> int {
    const int v = p.pages[rq.page_start + min(pi, rq.n_pages - 1)];
    return pi < item_pages ? v : -1;
  };
  constexpr int KB = SharedChunk<HD>::KBYTES, CB = SharedChunk<HD>::BYTES;
  constexpr int NLD = HD / 32;  // 16-byte loads per lane for a quarter chunk
  // waves 0 / 1: keys of the chunk's first / second page; 2 / 3: values
  auto gload = [&](u32x4 (&st)[NLD], int pid0, int pid1) {
    const int pg0 = (wave & 1) ? pid1 : pid0;
    const int pg = pg0 >= 0 ? pg0 : safe;  // past the end: masked, like the decode path
    const uint16_t* base = (wave < 2 ? p.k_pool : p.v_pool) + ((int64_t)pg * p.nkv + kvh) * (16 * HD);
#pragma unroll
    for (int i = 0; i < NLD; i++) st[i] = *reinterpret_cast<const u32x4*>(base + (i * 64 + lane) * 8);
  };
  auto swrite = [&](char* slot, const u32x4 (&st)[NLD]) {
#pragma unroll
    for (int i = 0; i < NLD; i++) {
      const int c = i * 64 + lane;
      char* dst;
      if (wave < 2) {
        const int key = 16 * (wave & 1) + c / (HD / 8), lc = c % (HD / 8);
        dst = slot + key * (HD * 2) + ((lc ^ ksw<HD>(key)) << 4);
      } else {
        const int d = c >> 1, lc = 2 * (wave & 1) + (c & 1);
        dst = slot + KB + d * 64 + ((lc ^ ((d >> 2) & 3)) << 4);
      }
      *reinterpret_cast<u32x4*>(dst) = st[i];
    }
  };
  // fragments of score block b (keys), or of output blocks DB0 .. (values)
  auto kread = [&](const char* slot, int b, u32x4 (&kf)[HD / 32]) {
#pragma unroll
    for (int ds = 0; ds < HD / 32; ds++) {
      const int key = 16 * (col >> 3) + 8 * ((col >> 2) & 1) + (col & 3) + 4 * b;
      kf[ds] = *reinterpret_cast<const u32x4*>(slot + key * (HD * 2) +
                                               (((4 * ds + g4) ^ ksw<HD>(key)) << 4));
    }
  };
  auto vread = [&](const char* slot, int db0, u32x4 (&vf)[HD / 32]) {
#pragma unroll
    for (int e = 0; e < HD / 32; e++) {
      const int d = 16 * (db0 + e) + col;
      vf[e] = *reinterpret_cast<const u32x4*>(slot + KB + d * 64 + ((g4 ^ ((d >> 2) & 3)) << 4));
    }
  };
  // Two register stagings used in turn: the loads of chunk kt + 2 are issued
  // while chunk kt is processed, and chunk kt + 1 (loaded during the previous
  // step) is then stored into the other LDS slot, which everyone finished
  // reading before the previous step's barrier; one barrier per chunk.  Page
  // ids are read one step ahead of their loads and issued before the step's
  // chunk loads: one counter tracks both, in order, so a wait for a page id
  // never waits for a chunk in flight.  Chunks past the tile's last one read
  // the request's first page and are never processed, so every step issues
  // the same loads.
  u32x4 sta[NLD], stb[NLD];
  int f0 = pid(4), f1 = pid(5);  // pages of the chunk the next step loads
  auto process = [&](int kt) {
    if (kt < wave_chunks) {
      // both row blocks from one read of the chunk's fragments, half a
      // chunk's keys (or values) at a time, each half applied to both
      // blocks before the next is read.  The wave's first row bounds both
      // blocks: the second block's rows come later.
      const char* slot = smem + (kt & 1) * CB;
      const int pi0 = 2 * kt;
      auto both = [&](auto mask) {
        constexpr bool MASK = decltype(mask)::value;
        f32x4 s1[2], s2[2];
#pragma unroll
        for (int b = 0; b < 2; b++) {
          u32x4 kf[HD / 32];
          kread(slot, b, kf);
          s1[b] = score_block<HD>(kf, qf);
          s2[b] = score_block<HD>(kf, qf2);
        }
        float sv1[2][4], sv2[2][4];
        const float mx1 = masked_scores<MASK>(s1, sv1, pi0, page_end, row_pos, g4);
        const float mx2 = masked_scores<MASK>(s2, sv2, pi0, page_end, row_pos2, g4);
        if (__any(mx1 > r1.thr || mx2 > r2.thr)) {
          raise_max(r1, mx1, p.scale_log2, inv_scale, o);
          raise_max(r2, mx2, p.scale_log2, inv_scale, o2);
        }
        const bf16x8 pb1 = probs(sv1, r1, p.scale_log2);
        const bf16x8 pb2 = probs(sv2, r2, p.scale_log2);
        uint32_t keep[4];
        value_keep(pi0, page_end, rq.kv_len, g4, keep);
        {
          u32x4 vf[HD / 32];
          vread(slot, 0, vf);
          values_part<HD, 0, HD / 32, MASK>(vf, o, pb1, keep);
          values_part<HD, 0, HD / 32, MASK>(vf, o2, pb2, keep);
        }
        {
          u32x4 vf[HD / 32];
          vread(slot, HD / 32, vf);
          values_part<HD, HD / 32, HD / 32, MASK>(vf, o, pb1, keep);
          values_part<HD, HD / 32, HD / 32, MASK>(vf, o2, pb2, keep);
        }
      };
      if (chunk_interior(pi0, page_end, wave_first_pos))
        both(std::integral_constant<bool, false>{});
      else
        both(std::integral_constant<bool, true>{});
    }
  };
  auto step = [&](int kt, u32x4 (&fill)[NLD], const u32x4 (&store)[NLD]) {
    const int g0 = pid(2 * kt + 6), g1 = pid(2 * kt + 7);  // for the next step
    __builtin_amdgcn_sched_barrier(0);
    gload(fill, f0, f1);  // chunk kt + 2
    __builtin_amdgcn_sched_barrier(0);
    f0 = g0;
    f1 = g1;
    process(kt);
    swrite(smem + ((kt + 1) & 1) * CB, store);  // chunk kt + 1
    __syncthreads();
  };
  {
    const int a0 = pid(0), a1 = pid(1), b0 = pid(2), b1 = pid(3);
    gload(sta, a0, a1);
    gload(stb, b0, b1);
  }
  swrite(smem, sta);
  __syncthreads();
  for (int kt = 0; kt < n_chunks; kt += 2) {
    step(kt, sta, stb);
    if (kt + 1 >= n_chunks) break;
    step(kt + 1, stb, sta);
  }
  // the rows' sums over their four lane groups (every lane takes part)
  const float l1 = lane_groups_sum(r1.l), l2 = lane_groups_sum(r2.l);
  if (row_valid) {
    const float inv = 1.f / l1;
    uint16_t* op = p.out + qtok * p.out_tok_stride + (int64_t)qhead * HD + 4 * g4;
#pragma unroll
    for (int db = 0; db < HD / 16; db++) {
      u32x2 w;
      w[0] = pack_bf16x2(o[db][0] * inv, o[db][1] * inv);
      w[1] = pack_bf16x2(o[db][2] * inv, o[db][3] * inv);
      *reinterpret_cast<u32x2*>(op + db * 16) = w;
    }
  }
  if (row_valid2) {
    const float inv = 1.f / l2;
    uint16_t* op = p.out + qtok2 * p.out_tok_stride + (int64_t)qhead * HD + 4 * g4;
#pragma unroll
    for (int db = 0; db < HD / 16; db++) {
      u32x2 w;
      w[0] = pack_bf16x2(o2[db][0] * inv, o2[db][1] * inv);
      w[1] = pack_bf16x2(o2[db][2] * inv, o2[db][3] * inv);
      *reinterpret_cast<u32x2*>(op + db * 16) = w;
    }
  }
}

// Decode item: the q heads it.head .. it.head + nrows - 1 (one per lane row)
// of the request's single token, over pages it.start .. of its table; the four
// waves stride over the split's 32-key chunks and combine through LDS.
template <int HD>
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
    load_chunk<HD>(ca, p, kvh, pid(pi), pid(pi + 1), safe, col, g4);
    while (true) {
      int pn = pi + chunk_step;
      if (pn >= page_end) {
        proc(ca, pi);
        break;
      }
      int nn0 = pid(pn + chunk_step), nn1 = pid(pn + chunk_step + 1);
      load_chunk<HD>(cb, p, kvh, n0, n1, safe, col, g4);
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
      load_chunk<HD>(ca, p, kvh, n0, n1, safe, col, g4);
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
    uint16_t* op = p.out + qtok * p.out_tok_stride + (int64_t)h * HD + dseg;
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
  else
    decode_item<HD>(p, it, rq, smem);
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
  p.out[(int64_t)rq.tok_start * p.out_tok_stride + (int64_t)h * HD + d] = f32_to_bf16(acc / L);
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
