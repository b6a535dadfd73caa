// mx_abi.cpp -- host side of libmx: argument validation, batch planning,
// metadata upload and the orchestration of the gfx950 kernels behind the C ABI
// declared in include/mx.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "mx.h"
#include "mx_kernels.h"

#define MX_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

using namespace mx;

thread_local std::string g_err;

mx_status fail(mx_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

mx_status hip_fail(hipError_t e, const char* what) {
  return fail(MX_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ------------------------------------------------------------------ validation
mx_status validate_shape(const mx_attn_shape* s) {
  if (!s) return fail(MX_ERR_NULL, "attention shape is NULL");
  if (s->n_q_heads <= 0 || s->n_kv_heads <= 0)
    return fail(MX_ERR_INVALID, "head counts must be positive (nq=%d, nkv=%d)", s->n_q_heads,
                s->n_kv_heads);
  if (s->n_q_heads % s->n_kv_heads != 0)
    return fail(MX_ERR_INVALID, "n_q_heads %d is not a multiple of n_kv_heads %d", s->n_q_heads,
                s->n_kv_heads);
  if (s->n_q_heads > 32767) return fail(MX_ERR_UNSUPPORTED, "more than 32767 q heads");
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(MX_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", s->head_dim);
  if (s->page_size != 16) return fail(MX_ERR_UNSUPPORTED, "page_size %d not supported (16)", s->page_size);
  if (s->pool_pages <= 0) return fail(MX_ERR_INVALID, "pool_pages must be positive");
  if (!(s->scale >= 0.f) || std::isinf(s->scale)) return fail(MX_ERR_INVALID, "invalid scale");
  return MX_OK;
}

mx_status validate_batch(const mx_batch* b, const mx_attn_shape* s, int64_t* T_out) {
  if (!b) return fail(MX_ERR_NULL, "batch is NULL");
  mx_status st = validate_shape(s);
  if (st != MX_OK) return st;
  if (b->num_reqs < 0) return fail(MX_ERR_INVALID, "num_reqs %d < 0", b->num_reqs);
  if (b->num_reqs > 0 && !b->reqs) return fail(MX_ERR_NULL, "reqs is NULL");
  int64_t T = 0;
  std::vector<int64_t> slots;
  for (int r = 0; r < b->num_reqs; r++) T += std::max(b->reqs[r].n_new, 0);
  slots.reserve((size_t)std::min<int64_t>(T, INT32_MAX / 2));
  T = 0;
  for (int r = 0; r < b->num_reqs; r++) {
    const mx_request& q = b->reqs[r];
    if (q.phase != MX_PREFILL && q.phase != MX_DECODE)
      return fail(MX_ERR_INVALID, "request %d: bad phase %d", r, q.phase);
    if (q.n_new < 1) return fail(MX_ERR_INVALID, "request %d: n_new %d < 1", r, q.n_new);
    if (q.ctx_len < 0) return fail(MX_ERR_INVALID, "request %d: ctx_len %d < 0", r, q.ctx_len);
    if (q.phase == MX_DECODE && (q.n_new != 1 || q.ctx_len < 1))
      return fail(MX_ERR_INVALID, "request %d: a decode needs n_new == 1 and ctx_len >= 1", r);
    const int64_t kv_len = (int64_t)q.ctx_len + q.n_new;
    if (kv_len > (int64_t)INT32_MAX - 16) return fail(MX_ERR_TOO_LARGE, "request %d: context too long", r);
    const int64_t need = ceil_div(kv_len, 16);
    if (q.n_pages < need)
      return fail(MX_ERR_NO_SPACE, "request %d: %d pages for %lld tokens (need %lld)", r, q.n_pages,
                  (long long)kv_len, (long long)need);
    if (!q.pages) return fail(MX_ERR_NULL, "request %d: pages is NULL", r);
    for (int i = 0; i < q.n_pages; i++)
      if (q.pages[i] < 0 || q.pages[i] >= s->pool_pages)
        return fail(MX_ERR_INVALID, "request %d: page id %d outside [0, %lld)", r, q.pages[i],
                    (long long)s->pool_pages);
    for (int i = 0; i < q.n_new; i++) {
      const int64_t p = (int64_t)q.ctx_len + i;
      slots.push_back((int64_t)q.pages[p / 16] * 16 + p % 16);
    }
    T += q.n_new;
    if (T > INT32_MAX / 2) return fail(MX_ERR_TOO_LARGE, "too many tokens");
  }
  std::sort(slots.begin(), slots.end());
  for (size_t i = 1; i < slots.size(); i++)
    if (slots[i] == slots[i - 1])
      return fail(MX_ERR_INVALID, "two new tokens write the same KV slot %lld", (long long)slots[i]);
  if (T_out) *T_out = T;
  return MX_OK;
}

mx_status validate_cfg(const mx_layer_cfg* c) {
  if (!c) return fail(MX_ERR_NULL, "layer cfg is NULL");
  mx_status st = validate_shape(&c->attn);
  if (st != MX_OK) return st;
  if (c->hidden <= 0 || c->hidden % 64)
    return fail(MX_ERR_UNSUPPORTED, "hidden %d must be a positive multiple of 64", c->hidden);
  if (c->ffn <= 0 || c->ffn % 64)
    return fail(MX_ERR_UNSUPPORTED, "ffn %d must be a positive multiple of 64", c->ffn);
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f))
    return fail(MX_ERR_INVALID, "invalid rms_eps or rope_theta");
  return MX_OK;
}

// ------------------------------------------------------------------ planning
constexpr int kXcds = 8;  // accelerator dies: workgroup b runs on die b % 8

struct Plan {
  int R = 0, T = 0;
  std::vector<ReqDev> reqs;
  std::vector<int32_t> pages;
  std::vector<AttnItem> items;
  std::vector<MergeItem> merges;
  int64_t n_parts = 0;
  int split_pages = 16;
  int group = 1;
  bool has_prefill = false;  // some work item is a prefill tile
};

// Decode splits: about 1024 work items (the chip holds 512 attention
// workgroups at once), at least 8 pages (four waves x two pages) per split.
// Fewer, longer items pay the start of an item (item, request and page-table
// reads before its first keys arrive) less often, and a request that fits in
// one split needs no partials and no merge: 2048 items were 3% slower on every
// layer shape, 512 no faster.
int choose_split_pages(const mx_batch* b, const mx_attn_shape* s) {
  const int group = s->n_q_heads / s->n_kv_heads;
  const int64_t sub = s->n_kv_heads * ceil_div(group, 16);
  int64_t total = 0;
  for (int r = 0; r < b->num_reqs; r++)
    if (b->reqs[r].phase == MX_DECODE)
      total += ceil_div((int64_t)b->reqs[r].ctx_len + 1, 16) * sub;
  const int64_t target_items = 1024;
  int64_t sp = ceil_div(std::max<int64_t>(total, 1), target_items);
  sp = std::max<int64_t>(8, std::min<int64_t>(sp, 4096));
  sp = (sp + 1) / 2 * 2;
  return (int)sp;
}

void build_plan(const mx_batch* b, const mx_attn_shape* s, bool with_items, Plan& p) {
  p.R = b->num_reqs;
  p.group = s->n_q_heads / s->n_kv_heads;
  p.split_pages = choose_split_pages(b, s);
  p.reqs.resize(p.R);
  int tok = 0, pg = 0;
  for (int r = 0; r < p.R; r++) {
    const mx_request& q = b->reqs[r];
    ReqDev& d = p.reqs[r];
    d.tok_start = tok;
    d.n_new = q.n_new;
    d.ctx_len = q.ctx_len;
    d.kv_len = q.ctx_len + q.n_new;
    d.page_start = pg;
    d.n_pages = (int)ceil_div(d.kv_len, 16);
    d.phase = q.phase;
    d.n_split = 1;
    tok += q.n_new;
    pg += d.n_pages;
  }
  p.T = tok;
  p.pages.resize(pg);
  for (int r = 0; r < p.R; r++)
    std::copy(b->reqs[r].pages, b->reqs[r].pages + p.reqs[r].n_pages,
              p.pages.begin() + p.reqs[r].page_start);
  if (!with_items) return;
  const int nq = s->n_q_heads;
  // prefill q tiles (heaviest work first: later tiles see more keys)
  for (int r = 0; r < p.R; r++) {
    const ReqDev& d = p.reqs[r];
    if (d.phase != MX_PREFILL) continue;
    const int tiles = (int)ceil_div(d.n_new, kPrefillTileRows);
    for (int qt = tiles - 1; qt >= 0; qt--)
      for (int h = 0; h < nq; h++) {
        AttnItem it;
        it.req = r;
        it.head = (int16_t)h;
        it.kind = 1;
        it.nrows = 16;
        it.start = qt * kPrefillTileRows;
        it.part = 0;
        p.items.push_back(it);
      }
  }
  // the hardware hands workgroups to free slots in list order, so the longest
  // items must not be left for the end: prefill tiles by the keys their last
  // rows scan, and the decode splits by page count, each longest first
  auto longer = [&](const AttnItem& a, const AttnItem& b) {
    const ReqDev& ra = p.reqs[a.req];
    const ReqDev& rb = p.reqs[b.req];
    return ra.ctx_len + std::min(a.start + kPrefillTileRows, ra.n_new) >
           rb.ctx_len + std::min(b.start + kPrefillTileRows, rb.n_new);
  };
  // (one prompt's tiles are generated in this order already)
  if (!std::is_sorted(p.items.begin(), p.items.end(), longer))
    std::stable_sort(p.items.begin(), p.items.end(), longer);
  // decode splits, longest first: a stable counting sort on the split's page
  // count (1 .. split_pages), so equal lengths keep request, split and head order
  std::vector<AttnItem> dec;
  std::vector<int64_t> count(p.split_pages + 2, 0);
  for (int r = 0; r < p.R; r++) {
    ReqDev& d = p.reqs[r];
    if (d.phase != MX_DECODE) continue;
    const int ns = (int)ceil_div(d.n_pages, p.split_pages);
    d.n_split = ns;
    int64_t part_base = 0;
    if (ns > 1) {
      part_base = p.n_parts;
      p.n_parts += (int64_t)nq * ns;
      p.merges.push_back(MergeItem{r, (int32_t)part_base});
    }
    for (int sp = 0; sp < ns; sp++) {
      const int len = std::min(p.split_pages, d.n_pages - sp * p.split_pages);
      for (int g = 0; g < s->n_kv_heads; g++)
        for (int h0 = 0; h0 < p.group; h0 += 16) {
          AttnItem it;
          it.req = r;
          it.head = (int16_t)(g * p.group + h0);
          it.kind = 0;
          it.nrows = (int8_t)std::min(16, p.group - h0);
          it.start = sp * p.split_pages;
          it.part = (int32_t)(part_base + (int64_t)it.head * ns + sp);
          dec.push_back(it);
          count[p.split_pages - len + 1]++;
        }
    }
  }
  for (size_t i = 1; i < count.size(); i++) count[i] += count[i - 1];
  std::vector<AttnItem> dsorted(dec.size());
  for (const AttnItem& it : dec) {
    const int len = std::min(p.split_pages, p.reqs[it.req].n_pages - it.start);
    dsorted[count[p.split_pages - len]++] = it;
  }
  // Prefill tiles (matrix-core bound) and decode splits (bound by HBM) are
  // interleaved in proportion to their counts, each list keeping its own
  // order: a CU then mostly holds one workgroup of each kind, whose demands
  // overlap, instead of all prefill tiles and then all decode splits.  At the
  // 70B shape with an 8192-token chunk the launch took 2.39 ms this way
  // against 2.83 ms with the prefill tiles first (and 2.85 ms with the decode
  // splits first).  The interleave runs per XCD: workgroup b runs on XCD
  // b % kXcds, so list position kXcds j + x is item j of XCD x's list, which
  // holds the prefill tiles of the KV heads h with h % kXcds == x and every
  // kXcds-th decode split.  The tiles of one KV head then read its keys and
  // values through one L2 instead of all eight, which leaves more of the
  // fabric to the decode stream beside them: the 70B launch at P = 8192 took
  // 2.10 ms against 2.24 ms with one list for all XCDs (same at P <= 4096).
  p.has_prefill = !p.items.empty();
  const std::vector<AttnItem> pre(std::move(p.items));
  const size_t nP = pre.size(), nD = dsorted.size();
  p.items.clear();
  p.items.reserve(nP + nD);
  auto interleave = [](const std::vector<AttnItem>& a, const std::vector<AttnItem>& b,
                       std::vector<AttnItem>& out) {
    for (size_t i = 0, j = 0; i < a.size() || j < b.size();) {
      // the list that is behind in its fraction done goes next
      if (j >= b.size() || (i < a.size() && (double)i * b.size() <= (double)j * a.size()))
        out.push_back(a[i++]);
      else
        out.push_back(b[j++]);
    }
  };
  if (nP == 0 || nD == 0) {
    interleave(pre, dsorted, p.items);
    return;
  }
  std::vector<AttnItem> px[kXcds], dx[kXcds], sub[kXcds];
  for (const AttnItem& it : pre) px[(it.head / p.group) % kXcds].push_back(it);
  for (size_t j = 0; j < nD; j++) dx[j % kXcds].push_back(dsorted[j]);
  size_t longest = 0;
  for (int x = 0; x < kXcds; x++) {
    interleave(px[x], dx[x], sub[x]);
    longest = std::max(longest, sub[x].size());
  }
  for (size_t j = 0; j < longest; j++)
    for (int x = 0; x < kXcds; x++)
      if (j < sub[x].size()) p.items.push_back(sub[x][j]);
}

// ------------------------------------------------------------------ workspace layout
struct Layout {
  size_t reqs = 0, pages = 0, items = 0, merges = 0, inv_freq = 0, meta_end = 0;
  size_t tok_req = 0, tok_pos = 0, tok_slot = 0, rope_cs = 0;
  size_t part_o = 0, part_ml = 0;
  size_t h = 0, q = 0, o = 0, x1 = 0, a = 0, scratch = 0, scratch_floats = 0;
  size_t total = 0;
};

size_t gemm_scratch_bound(const mx_layer_cfg* c, int64_t T) {
  const int H = c->hidden, F = c->ffn, nq = c->attn.n_q_heads, nkv = c->attn.n_kv_heads,
            d = c->attn.head_dim;
  const int M = (int)T;
  size_t m = gemm_scratch_floats(M, (nq + 2 * nkv) * d, H);
  m = std::max(m, gemm_scratch_floats(M, H, nq * d));
  m = std::max(m, gemm_scratch_floats(M, 2 * F, H));
  m = std::max(m, gemm_scratch_floats(M, H, F));
  return m;
}

Layout make_layout(int64_t R, int64_t T, int64_t n_pages, int64_t n_items, int64_t n_merges,
                   int64_t n_parts, const mx_attn_shape* s, const mx_layer_cfg* c,
                   size_t scratch_floats) {
  Layout L;
  size_t o = 0;
  const int d = s->head_dim;
  L.reqs = o; o = align_up(o + R * sizeof(ReqDev));
  L.pages = o; o = align_up(o + n_pages * sizeof(int32_t));
  L.items = o; o = align_up(o + n_items * sizeof(AttnItem));
  L.merges = o; o = align_up(o + n_merges * sizeof(MergeItem));
  L.inv_freq = o; o = align_up(o + (d / 2) * sizeof(double));
  L.meta_end = o;
  L.tok_req = o; o = align_up(o + T * 4);
  L.tok_pos = o; o = align_up(o + T * 4);
  L.tok_slot = o; o = align_up(o + T * 8);
  L.part_o = o; o = align_up(o + n_parts * d * 4);
  L.part_ml = o; o = align_up(o + n_parts * 8);
  if (c) {
    const int64_t H = c->hidden, F = c->ffn, nq = s->n_q_heads;
    // h, o and a are projection inputs in the tile layout (whole tile rows)
    L.rope_cs = o; o = align_up(o + T * (d / 2) * 8);
    L.h = o; o = align_up(o + tile_elems(T, H) * 2);
    L.q = o; o = align_up(o + T * nq * d * 2);
    L.o = o; o = align_up(o + tile_elems(T, nq * d) * 2);
    L.x1 = o; o = align_up(o + T * H * 2);
    L.a = o; o = align_up(o + tile_elems(T, F) * 2);
    L.scratch = o; o = align_up(o + scratch_floats * 4);
    L.scratch_floats = scratch_floats;
  }
  L.total = o;
  return L;
}

Layout layout_for(const Plan& p, const mx_attn_shape* s, const mx_layer_cfg* c) {
  const size_t sc = c ? gemm_scratch_bound(c, p.T) : 0;
  return make_layout(p.R, p.T, (int64_t)p.pages.size(), (int64_t)p.items.size(),
                     (int64_t)p.merges.size(), p.n_parts, s, c, sc);
}

// ------------------------------------------------------------------ per-device state
// Metadata staging: kRing pinned host buffers used in turn.  A buffer may be
// rewritten once the upload that read it has run.  A completion event costs
// the stream a few microseconds, so on the null stream one is recorded per
// group of up to kEvery consecutive uploads, after the group's last upload,
// and covers the whole group: a group ends after kEvery uploads, at the last
// buffer of the ring, or when the next upload is on another stream.  On any
// other stream every upload closes its own group in the same call: an event is
// never recorded on a stream the caller may have destroyed since (the null
// stream cannot be).  A group never wraps around the ring, so the event that
// covers buffer i was recorded into a buffer at or after i, which is not
// reused (and so not re-recorded) before i.
struct DeviceState {
  std::mutex mu;
  bool init = false;
  static constexpr int kRing = 8;
  static constexpr int kEvery = 4;
  void* buf[kRing] = {};   // pinned host staging buffers
  void* dbuf[kRing] = {};  // the same buffers as the device reads them
  size_t cap[kRing] = {};
  hipEvent_t ev[kRing] = {};
  bool used[kRing] = {};
  int cover[kRing] = {};   // buffer whose event covers this buffer's last upload
  int next = 0;
  int group_first = -1;    // first buffer of the open group (-1: none)
  hipStream_t group_stream = nullptr;
};

std::mutex g_dev_mu;
std::map<int, DeviceState*> g_devs;

mx_status device_state(DeviceState** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  DeviceState* ds;
  {
    std::lock_guard<std::mutex> g(g_dev_mu);
    auto it = g_devs.find(dev);
    if (it == g_devs.end()) {
      ds = new DeviceState();
      g_devs[dev] = ds;
    } else {
      ds = it->second;
    }
  }
  std::lock_guard<std::mutex> g(ds->mu);
  if (!ds->init) {
    e = gemm_init();
    if (e != hipSuccess) return hip_fail(e, "kernel attribute setup");
    for (int i = 0; i < DeviceState::kRing; i++) {
      e = hipEventCreateWithFlags(&ds->ev[i], hipEventDisableTiming);
      if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    }
    ds->init = true;
  }
  *out = ds;
  return MX_OK;
}

// Packs the plan's metadata into a pinned staging buffer and enqueues its copy
// into the workspace (a kernel that reads the buffer through its device
// mapping).  A staging slot is rewritten or freed only after the event
// recorded behind its previous copy has completed.
// Records the open group's event after its last upload (buffer `last`) on the
// group's stream; every buffer of the group is then covered by it.
hipError_t close_group(DeviceState* ds, int last) {
  hipError_t e = hipEventRecord(ds->ev[last], ds->group_stream);
  if (e != hipSuccess) return e;
  for (int j = ds->group_first;; j = (j + 1) % DeviceState::kRing) {
    ds->cover[j] = last;
    if (j == last) break;
  }
  ds->group_first = -1;
  return hipSuccess;
}

// The metadata block [0, L.meta_end) of the workspace, as the kernels read it:
// request records, page tables, attention work items, merge items, rotary
// inverse frequencies.
void pack_meta(const Plan& p, const Layout& L, const mx_attn_shape* s, float theta, char* h) {
  memset(h, 0, L.meta_end);
  if (!p.reqs.empty()) memcpy(h + L.reqs, p.reqs.data(), p.reqs.size() * sizeof(ReqDev));
  if (!p.pages.empty()) memcpy(h + L.pages, p.pages.data(), p.pages.size() * sizeof(int32_t));
  if (!p.items.empty()) memcpy(h + L.items, p.items.data(), p.items.size() * sizeof(AttnItem));
  if (!p.merges.empty()) memcpy(h + L.merges, p.merges.data(), p.merges.size() * sizeof(MergeItem));
  double* inv = (double*)(h + L.inv_freq);
  const int d = s->head_dim;
  for (int k = 0; k < d / 2; k++) inv[k] = std::pow((double)theta, -2.0 * k / d);
}

mx_status upload_meta(const Plan& p, const Layout& L, const mx_attn_shape* s, float theta,
                      void* ws, hipStream_t stream) {
  DeviceState* ds;
  mx_status st = device_state(&ds);
  if (st != MX_OK) return st;
  std::lock_guard<std::mutex> g(ds->mu);
  const int i = ds->next;
  ds->next = (ds->next + 1) % DeviceState::kRing;
  hipError_t e;
  // the open group is on another stream: close it there first
  if (ds->group_first >= 0 && ds->group_stream != stream) {
    if ((e = close_group(ds, (i + DeviceState::kRing - 1) % DeviceState::kRing)) != hipSuccess)
      return hip_fail(e, "hipEventRecord");
  }
  if (ds->used[i]) {
    e = hipEventSynchronize(ds->ev[ds->cover[i]]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  }
  if (ds->cap[i] < L.meta_end) {
    if (ds->buf[i]) {
      e = hipHostFree(ds->buf[i]);
      ds->buf[i] = ds->dbuf[i] = nullptr;
      ds->cap[i] = 0;
      if (e != hipSuccess) return hip_fail(e, "hipHostFree");
    }
    const size_t cap = std::max<size_t>(L.meta_end * 2, 1 << 16);
    e = hipHostMalloc(&ds->buf[i], cap, hipHostMallocMapped);
    if (e != hipSuccess) { ds->buf[i] = nullptr; ds->cap[i] = 0; return hip_fail(e, "hipHostMalloc"); }
    e = hipHostGetDevicePointer(&ds->dbuf[i], ds->buf[i], 0);
    if (e != hipSuccess) {
      (void)hipHostFree(ds->buf[i]);  // the lookup's error is the one reported
      ds->buf[i] = ds->dbuf[i] = nullptr;
      ds->cap[i] = 0;
      return hip_fail(e, "hipHostGetDevicePointer");
    }
    ds->cap[i] = cap;
  }
  pack_meta(p, L, s, theta, (char*)ds->buf[i]);
  e = launch_upload(ds->dbuf[i], ws, L.meta_end, stream);
  if (e != hipSuccess) return hip_fail(e, "metadata upload launch");
  ds->used[i] = true;
  if (ds->group_first < 0) {
    ds->group_first = i;
    ds->group_stream = stream;
  }
  const int size = i - ds->group_first + 1;
  if (stream != nullptr || size == DeviceState::kEvery || i == DeviceState::kRing - 1) {
    if ((e = close_group(ds, i)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  return MX_OK;
}

template <typename T>
T* at(void* ws, size_t off) { return reinterpret_cast<T*>((char*)ws + off); }

float eff_scale(const mx_attn_shape* s) {
  return s->scale > 0.f ? s->scale : 1.0f / std::sqrt((float)s->head_dim);
}

AttnParams attn_params(const Plan& p, const Layout& L, const mx_attn_shape* s, void* ws,
                       const uint16_t* q, int64_t q_stride, const uint16_t* kp,
                       const uint16_t* vp, uint16_t* out) {
  AttnParams a;
  a.q = q;
  a.q_tok_stride = q_stride;
  a.k_pool = kp;
  a.v_pool = vp;
  a.out = out;
  a.out_tok_stride = (int64_t)s->n_q_heads * s->head_dim;
  a.out_tiled = 0;
  a.reqs = at<ReqDev>(ws, L.reqs);
  a.pages = at<int32_t>(ws, L.pages);
  a.items = at<AttnItem>(ws, L.items);
  a.part_o = at<float>(ws, L.part_o);
  a.part_ml = at<float>(ws, L.part_ml);
  a.nq = s->n_q_heads;
  a.nkv = s->n_kv_heads;
  a.group = p.group;
  a.split_pages = p.split_pages;
  a.scale_log2 = eff_scale(s) * 1.4426950408889634f;
  a.decode_only = p.has_prefill ? 0 : 1;
  return a;
}

// packed weight regions
struct WLayout {
  size_t g1, qkv, o, g2, gu, down, total;
};
WLayout wlayout(const mx_layer_cfg* c) {
  const size_t H = c->hidden, F = c->ffn, nq = c->attn.n_q_heads, nkv = c->attn.n_kv_heads,
               d = c->attn.head_dim;
  WLayout w;
  size_t o = 0;
  w.g1 = o; o = align_up(o + H * 2);
  w.qkv = o; o = align_up(o + (nq + 2 * nkv) * d * H * 2);
  w.o = o; o = align_up(o + H * nq * d * 2);
  w.g2 = o; o = align_up(o + H * 2);
  w.gu = o; o = align_up(o + 2 * F * H * 2);
  w.down = o; o = align_up(o + H * F * 2);
  w.total = o;
  return w;
}

// ------------------------------------------------------------------ launch timing
// Optional per-launch timing (hipEvents recorded on the caller's stream around
// each kernel launch).  Off by default; costs two event records per launch.
struct Profiler {
  std::mutex mu;
  bool on = false;
  struct Rec {
    const char* name;
    hipEvent_t a, b;
  };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> free_events;
  std::vector<const char*> names;
  std::vector<double> total_ms;
  std::vector<int> counts;

  hipEvent_t get() {
    if (!free_events.empty()) {
      hipEvent_t e = free_events.back();
      free_events.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};
Profiler g_prof;

template <typename F>
hipError_t timed(const char* name, hipStream_t stream, F&& launch) {
  bool on;
  {
    std::lock_guard<std::mutex> g(g_prof.mu);
    on = g_prof.on;
  }
  if (!on) return launch();
  hipEvent_t a, b;
  {
    std::lock_guard<std::mutex> g(g_prof.mu);
    a = g_prof.get();
    b = g_prof.get();
  }
  if (!a || !b) return launch();
  hipError_t e = hipEventRecord(a, stream);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, stream);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> g(g_prof.mu);
  g_prof.pending.push_back({name, a, b});
  return hipSuccess;
}

}  // namespace

// ======================================================================= ABI
MX_EXPORT const char* mx_status_str(mx_status s) {
  switch (s) {
    case MX_OK: return "MX_OK";
    case MX_ERR_INVALID: return "MX_ERR_INVALID";
    case MX_ERR_NO_SPACE: return "MX_ERR_NO_SPACE";
    case MX_ERR_TOO_LARGE: return "MX_ERR_TOO_LARGE";
    case MX_ERR_UNSUPPORTED: return "MX_ERR_UNSUPPORTED";
    case MX_ERR_NULL: return "MX_ERR_NULL";
    case MX_ERR_HIP: return "MX_ERR_HIP";
  }
  return "MX_ERR_UNKNOWN";
}

MX_EXPORT const char* mx_last_error(void) { return g_err.c_str(); }

MX_EXPORT uint32_t mx_version(void) { return (1u << 16) | 0u; }

// Device tensors are read and written with 16-byte vector accesses.
static mx_status check_aligned(std::initializer_list<const void*> ptrs) {
  for (const void* q : ptrs)
    if ((uintptr_t)q & 15) return fail(MX_ERR_INVALID, "device pointer %p is not 16-byte aligned", q);
  return MX_OK;
}

MX_EXPORT mx_status mx_batch_validate(const mx_batch* batch, const mx_attn_shape* shape) {
  g_err.clear();
  return validate_batch(batch, shape, nullptr);
}

MX_EXPORT size_t mx_workspace_bytes_for(const mx_batch* batch, const mx_attn_shape* shape,
                                        const mx_layer_cfg* cfg) {
  g_err.clear();
  if (cfg) {
    if (validate_cfg(cfg) != MX_OK) return 0;
    shape = &cfg->attn;
  }
  if (validate_batch(batch, shape, nullptr) != MX_OK) return 0;
  Plan p;
  build_plan(batch, shape, true, p);
  return layout_for(p, shape, cfg).total;
}

MX_EXPORT size_t mx_workspace_bytes(const mx_layer_cfg* cfg, const mx_attn_shape* shape,
                                    int32_t max_tokens, int32_t max_reqs, int64_t max_pages) {
  g_err.clear();
  if (cfg) {
    if (validate_cfg(cfg) != MX_OK) return 0;
    shape = &cfg->attn;
  } else if (validate_shape(shape) != MX_OK) {
    return 0;
  }
  if (max_tokens < 0 || max_reqs < 0 || max_pages < 0) {
    fail(MX_ERR_INVALID, "negative bound");
    return 0;
  }
  const int64_t nq = shape->n_q_heads, nkv = shape->n_kv_heads, group = nq / nkv;
  // every split has at least 8 pages, so splits <= pages / 8 + requests
  const int64_t splits = max_pages / 8 + max_reqs;
  const int64_t items =
      splits * nkv * ceil_div(group, 16) + (max_tokens / kPrefillTileRows + max_reqs) * nq;
  const int64_t parts = splits * nq;
  const size_t scratch = cfg ? kMaxSplitFloats : 0;
  return make_layout(max_reqs, max_tokens, max_pages, items, max_reqs, parts, shape, cfg, scratch)
      .total;
}

MX_EXPORT size_t mx_packed_weights_bytes(const mx_layer_cfg* cfg) {
  g_err.clear();
  if (validate_cfg(cfg) != MX_OK) return 0;
  return wlayout(cfg).total;
}

MX_EXPORT mx_status mx_pack_weights(const mx_layer_cfg* cfg, const mx_layer_weights* w,
                                    void* packed, size_t packed_bytes, hipStream_t stream) {
  g_err.clear();
  mx_status st = validate_cfg(cfg);
  if (st != MX_OK) return st;
  if (!w || !packed || !w->ln1_g || !w->w_qkv || !w->w_o || !w->ln2_g || !w->w_gate_up || !w->w_down)
    return fail(MX_ERR_NULL, "weight pointer is NULL");
  if ((st = check_aligned({packed, w->ln1_g, w->w_qkv, w->w_o, w->ln2_g, w->w_gate_up, w->w_down})) !=
      MX_OK)
    return st;
  const WLayout L = wlayout(cfg);
  if (packed_bytes < L.total)
    return fail(MX_ERR_TOO_LARGE, "packed buffer %zu bytes < %zu", packed_bytes, L.total);
  DeviceState* ds;
  st = device_state(&ds);
  if (st != MX_OK) return st;
  const size_t H = cfg->hidden, F = cfg->ffn, nq = cfg->attn.n_q_heads,
               nkv = cfg->attn.n_kv_heads, d = cfg->attn.head_dim;
  char* P = (char*)packed;
  hipError_t e;
#define MX_CP(off, src, bytes)                                                        \
  e = hipMemcpyAsync(P + (off), (src), (bytes), hipMemcpyDeviceToDevice, stream);    \
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (pack)");
  MX_CP(L.g1, w->ln1_g, H * 2)
  MX_CP(L.g2, w->ln2_g, H * 2)
#undef MX_CP
  // the four matrices in the GEMMs' tiled layout (row permutation applied on the way)
#define MX_TILE(off, src, N, K, kind, what)                                                      \
  e = launch_pack_tiled((src), (uint16_t*)(P + (off)), (int)(N), (int)(K), (kind), (int)nq,      \
                        (int)nkv, (int)d, (int)F, stream);                                       \
  if (e != hipSuccess) return hip_fail(e, what);
  MX_TILE(L.qkv, w->w_qkv, (nq + 2 * nkv) * d, H, 1, "qkv packing launch")
  MX_TILE(L.o, w->w_o, H, nq * d, 0, "o packing launch")
  MX_TILE(L.gu, w->w_gate_up, 2 * F, H, 2, "gate/up packing launch")
  MX_TILE(L.down, w->w_down, H, F, 0, "down packing launch")
#undef MX_TILE
  return MX_OK;
}

static mx_status check_ws(const Layout& L, void* ws, size_t ws_bytes) {
  if (!ws) return fail(MX_ERR_NULL, "workspace is NULL");
  if (ws_bytes < L.total)
    return fail(MX_ERR_TOO_LARGE, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  return MX_OK;
}

MX_EXPORT mx_status mx_kv_append(const mx_batch* batch, const mx_attn_shape* shape,
                                 const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                                 uint16_t* v_pool, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err.clear();
  int64_t T;
  mx_status st = validate_batch(batch, shape, &T);
  if (st != MX_OK) return st;
  if (T == 0) return MX_OK;
  if (!k_new || !v_new || !k_pool || !v_pool) return fail(MX_ERR_NULL, "tensor pointer is NULL");
  if ((st = check_aligned({k_new, v_new, k_pool, v_pool, ws})) != MX_OK) return st;
  Plan p;
  build_plan(batch, shape, false, p);
  const Layout L = layout_for(p, shape, nullptr);
  if ((st = check_ws(L, ws, ws_bytes)) != MX_OK) return st;
  if ((st = upload_meta(p, L, shape, 1e4f, ws, stream)) != MX_OK) return st;
  hipError_t e = launch_token_map(at<ReqDev>(ws, L.reqs), p.R, p.T, at<int32_t>(ws, L.pages),
                                  at<int32_t>(ws, L.tok_req), at<int32_t>(ws, L.tok_pos),
                                  at<int64_t>(ws, L.tok_slot), nullptr, nullptr, 0, stream);
  if (e != hipSuccess) return hip_fail(e, "token map launch");
  e = launch_kv_append(k_new, v_new, k_pool, v_pool, at<int64_t>(ws, L.tok_slot), p.T,
                       shape->n_kv_heads, shape->head_dim, stream);
  if (e != hipSuccess) return hip_fail(e, "kv append launch");
  return MX_OK;
}

MX_EXPORT mx_status mx_paged_attn(const mx_batch* batch, const mx_attn_shape* shape,
                                  const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                                  uint16_t* out, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err.clear();
  int64_t T;
  mx_status st = validate_batch(batch, shape, &T);
  if (st != MX_OK) return st;
  if (T == 0) return MX_OK;
  if (!q || !k_pool || !v_pool || !out) return fail(MX_ERR_NULL, "tensor pointer is NULL");
  if ((st = check_aligned({q, k_pool, v_pool, out, ws})) != MX_OK) return st;
  Plan p;
  build_plan(batch, shape, true, p);
  const Layout L = layout_for(p, shape, nullptr);
  if ((st = check_ws(L, ws, ws_bytes)) != MX_OK) return st;
  if ((st = upload_meta(p, L, shape, 1e4f, ws, stream)) != MX_OK) return st;
  AttnParams a = attn_params(p, L, shape, ws, q, (int64_t)shape->n_q_heads * shape->head_dim,
                             k_pool, v_pool, out);
  hipError_t e = timed("paged_attn", stream, [&] {
    return launch_paged_attn(a, (int)p.items.size(), at<MergeItem>(ws, L.merges),
                             (int)p.merges.size(), shape->head_dim, stream);
  });
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  return MX_OK;
}

// ------------------------------------------------------------------ static scratch
// Device memory of mx_paged_attn_static: the metadata block and the split
// partials of one call, in a file-scope array of kStaticScratchBytes that
// every GPU the library runs on holds until the process ends.  Host code uses
// the array only through the device address hipGetSymbolAddress returns for
// the current device (the array's name is a host-side stand-in, not a device
// address); the address is taken once per device, on the entry point's first
// call there, and kept.
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptr;

// Host side of the same calls: the metadata block is packed into this
// file-scope buffer (no allocation per call) and copied from it with
// hipMemcpyAsync.  From pageable memory HIP performs that copy synchronously
// (the source has been read when the call returns), so the buffer is free
// again on return; the lock keeps the calls of different threads apart while
// they pack and copy.
std::mutex g_static_host_mu;
alignas(64) char g_static_host[kStaticScratchBytes];

mx_status static_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> g(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return MX_OK;
  }
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (static scratch)");
  if (!ptr) return fail(MX_ERR_HIP, "hipGetSymbolAddress returned NULL for the static scratch");
  g_scratch_ptr[dev] = ptr;
  *out = ptr;
  return MX_OK;
}

MX_EXPORT size_t mx_paged_attn_static_max_bytes(void) { return kStaticScratchBytes; }

MX_EXPORT mx_status mx_paged_attn_static(const mx_batch* batch, const mx_attn_shape* shape,
                                         const uint16_t* q, const uint16_t* k_pool,
                                         const uint16_t* v_pool, uint16_t* out,
                                         hipStream_t stream) {
  g_err.clear();
  int64_t T;
  mx_status st = validate_batch(batch, shape, &T);
  if (st != MX_OK) return st;
  if (T == 0) return MX_OK;
  if (!q || !k_pool || !v_pool || !out) return fail(MX_ERR_NULL, "tensor pointer is NULL");
  if ((st = check_aligned({q, k_pool, v_pool, out})) != MX_OK) return st;
  Plan p;
  build_plan(batch, shape, true, p);
  const Layout L = layout_for(p, shape, nullptr);
  if (L.total > kStaticScratchBytes)
    return fail(MX_ERR_TOO_LARGE,
                "batch needs %zu bytes of scratch; the static scratch holds %zu (use mx_paged_attn "
                "with a workspace)",
                L.total, kStaticScratchBytes);
  void* ws = nullptr;
  if ((st = static_scratch(&ws)) != MX_OK) return st;
  // the metadata block, packed on the host and copied into the scratch in
  // stream order (nothing in the scratch needs to start at zero: every split
  // partial is written by its item before the merge reads it)
  hipError_t e;
  {
    std::lock_guard<std::mutex> g(g_static_host_mu);
    pack_meta(p, L, shape, 1e4f, g_static_host);  // L.meta_end <= L.total, checked above
    e = hipMemcpyAsync(ws, g_static_host, L.meta_end, hipMemcpyHostToDevice, stream);
  }
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (metadata)");
  AttnParams a = attn_params(p, L, shape, ws, q, (int64_t)shape->n_q_heads * shape->head_dim,
                             k_pool, v_pool, out);
  e = timed("paged_attn", stream, [&] {
    return launch_paged_attn(a, (int)p.items.size(), at<MergeItem>(ws, L.merges),
                             (int)p.merges.size(), shape->head_dim, stream);
  });
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  return MX_OK;
}

MX_EXPORT mx_status mx_layer_step(const mx_batch* batch, const mx_layer_cfg* cfg,
                                  const void* packed_weights, const uint16_t* x, uint16_t* y,
                                  uint16_t* k_pool, uint16_t* v_pool, void* ws, size_t ws_bytes,
                                  hipStream_t stream) {
  g_err.clear();
  mx_status st = validate_cfg(cfg);
  if (st != MX_OK) return st;
  const mx_attn_shape* s = &cfg->attn;
  int64_t T;
  if ((st = validate_batch(batch, s, &T)) != MX_OK) return st;
  if (T == 0) return MX_OK;
  if (!packed_weights || !x || !y || !k_pool || !v_pool)
    return fail(MX_ERR_NULL, "tensor pointer is NULL");
  if (x == y) return fail(MX_ERR_INVALID, "y must not alias x");
  if ((st = check_aligned({packed_weights, x, y, k_pool, v_pool, ws})) != MX_OK) return st;
  Plan p;
  build_plan(batch, s, true, p);
  const Layout L = layout_for(p, s, cfg);
  if ((st = check_ws(L, ws, ws_bytes)) != MX_OK) return st;
  if ((st = upload_meta(p, L, s, cfg->rope_theta, ws, stream)) != MX_OK) return st;
  const WLayout W = wlayout(cfg);
  const char* P = (const char*)packed_weights;
  const int H = cfg->hidden, F = cfg->ffn, nq = s->n_q_heads, nkv = s->n_kv_heads,
            d = s->head_dim;
  const int Nqkv = (nq + 2 * nkv) * d;
  const int M = p.T;
  uint16_t* h = at<uint16_t>(ws, L.h);
  uint16_t* q = at<uint16_t>(ws, L.q);
  uint16_t* o = at<uint16_t>(ws, L.o);
  uint16_t* x1 = at<uint16_t>(ws, L.x1);
  uint16_t* act = at<uint16_t>(ws, L.a);
  float* scratch = at<float>(ws, L.scratch);
  float2* rope_cs = at<float2>(ws, L.rope_cs);
  hipError_t e;
#define MX_CK(call, what) \
  if ((e = (call)) != hipSuccess) return hip_fail(e, what);
  // a1 + a2: token map and rotary table, and RMSNorm 1, in one launch
  MX_CK(timed("token_map+rmsnorm_1", stream, [&] {
          return launch_prologue(at<ReqDev>(ws, L.reqs), p.R, p.T, at<int32_t>(ws, L.pages),
                                 at<int32_t>(ws, L.tok_req), at<int32_t>(ws, L.tok_pos),
                                 at<int64_t>(ws, L.tok_slot), at<double>(ws, L.inv_freq),
                                 rope_cs, d / 2, x, (const uint16_t*)(P + W.g1), h, H,
                                 cfg->rms_eps, stream);
        }), "prologue launch")
  // a3-a5: QKV projection with RoPE and the KV append fused into its epilogue
  {
    GemmArgs g{h, (const uint16_t*)(P + W.qkv), nullptr, nullptr, scratch, M, Nqkv, H, H, H, 0, 0, EPI_QKV,
               QkvEpilogue{rope_cs, at<int64_t>(ws, L.tok_slot), q, k_pool, v_pool, nq, nkv, d}};
    set_b_tiled(g);
    g.a_tiled = 1;
    MX_CK(timed("gemm_qkv", stream, [&] { return launch_gemm(g, L.scratch_floats, stream); }),
          "qkv gemm launch")
  }
  // a6: paged attention, prefill and decode rows in one launch (+ split merge)
  {
    AttnParams a = attn_params(p, L, s, ws, q, (int64_t)nq * d, k_pool, v_pool, o);
    a.out_tiled = 1;  // o feeds the output projection
    MX_CK(timed("paged_attn", stream, [&] {
            return launch_paged_attn(a, (int)p.items.size(), at<MergeItem>(ws, L.merges),
                                     (int)p.merges.size(), d, stream);
          }), "attention launch")
  }
  // a7 + a8: output projection + residual, then RMSNorm 2.  When (some rows
  // of) the projection are split over K, their reduce, the residual and the
  // norm of every row run as one kernel (timed as o_reduce+rmsnorm_2), which
  // reads the fp32 planes once and keeps each x1 row in registers for the norm.
  {
    GemmArgs g{o, (const uint16_t*)(P + W.o), x1, x, scratch, M, H, nq * d, nq * d, nq * d, H, H, EPI_RESIDUAL, {}};
    set_b_tiled(g);
    g.a_tiled = 1;
    const uint16_t* g2 = (const uint16_t*)(P + W.g2);
    const bool fuse = H <= kFusedNormMaxH;  // the fused kernel holds a row in registers
    int split_row = M, ks = 1;
    MX_CK(timed("gemm_o", stream, [&] {
            return fuse ? launch_gemm_unreduced(g, L.scratch_floats, &split_row, &ks, stream)
                        : launch_gemm(g, L.scratch_floats, stream);
          }), "o gemm launch")
    MX_CK(timed(ks > 1 ? "o_reduce+rmsnorm_2" : "rmsnorm_2", stream, [&] {
            return ks > 1 ? launch_reduce_residual_rmsnorm(scratch, ks, x, x1, g2, h, M, H,
                                                           cfg->rms_eps, split_row, stream)
                          : launch_rmsnorm(x1, g2, h, M, H, cfg->rms_eps, stream);
          }), "rmsnorm launch")
  }
  // a9: gate/up projection + SwiGLU
  {
    GemmArgs g{h, (const uint16_t*)(P + W.gu), act, nullptr, scratch, M, 2 * F, H, H, H, F, 0, EPI_SWIGLU, {}};
    set_b_tiled(g);
    g.a_tiled = 1;
    g.c_tiled = 1;  // act feeds the down projection
    MX_CK(timed("gemm_gate_up", stream, [&] { return launch_gemm(g, L.scratch_floats, stream); }),
          "gate/up gemm launch")
  }
  // a10: down projection + residual
  {
    GemmArgs g{act, (const uint16_t*)(P + W.down), y, x1, scratch, M, H, F, F, F, H, H, EPI_RESIDUAL, {}};
    set_b_tiled(g);
    g.a_tiled = 1;
    MX_CK(timed("gemm_down", stream, [&] { return launch_gemm(g, L.scratch_floats, stream); }),
          "down gemm launch")
  }
#undef MX_CK
  return MX_OK;
}

MX_EXPORT mx_status mx_layer_workspace_offsets(const mx_batch* batch, const mx_layer_cfg* cfg,
                                               size_t off[5]) {
  g_err.clear();
  mx_status st = validate_cfg(cfg);
  if (st != MX_OK) return st;
  if ((st = validate_batch(batch, &cfg->attn, nullptr)) != MX_OK) return st;
  if (!off) return fail(MX_ERR_NULL, "off is NULL");
  Plan p;
  build_plan(batch, &cfg->attn, true, p);
  const Layout L = layout_for(p, &cfg->attn, cfg);
  off[0] = L.h;
  off[1] = L.q;
  off[2] = L.o;
  off[3] = L.x1;
  off[4] = L.a;
  return MX_OK;
}

MX_EXPORT mx_status mx_debug_token_map(const mx_batch* batch, const mx_attn_shape* shape,
                                       int32_t* tok_req, int32_t* tok_pos, int64_t* tok_slot,
                                       void* ws, size_t ws_bytes, hipStream_t stream) {
  g_err.clear();
  int64_t T;
  mx_status st = validate_batch(batch, shape, &T);
  if (st != MX_OK) return st;
  if (T == 0) return MX_OK;
  if (!tok_req || !tok_pos || !tok_slot) return fail(MX_ERR_NULL, "output pointer is NULL");
  Plan p;
  build_plan(batch, shape, false, p);
  const Layout L = layout_for(p, shape, nullptr);
  if ((st = check_ws(L, ws, ws_bytes)) != MX_OK) return st;
  if ((st = upload_meta(p, L, shape, 1e4f, ws, stream)) != MX_OK) return st;
  hipError_t e = launch_token_map(at<ReqDev>(ws, L.reqs), p.R, p.T, at<int32_t>(ws, L.pages),
                                  at<int32_t>(ws, L.tok_req), at<int32_t>(ws, L.tok_pos),
                                  at<int64_t>(ws, L.tok_slot), nullptr, nullptr, 0, stream);
  if (e != hipSuccess) return hip_fail(e, "token map launch");
  e = hipMemcpyAsync(tok_req, at<int32_t>(ws, L.tok_req), T * 4, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(tok_pos, at<int32_t>(ws, L.tok_pos), T * 4, hipMemcpyDeviceToDevice, stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(tok_slot, at<int64_t>(ws, L.tok_slot), T * 8, hipMemcpyDeviceToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (token map)");
  return MX_OK;
}

MX_EXPORT mx_status mx_debug_gather(const mx_batch* batch, const mx_attn_shape* shape, int32_t req,
                                    const uint16_t* k_pool, const uint16_t* v_pool,
                                    uint16_t* k_out, uint16_t* v_out, void* ws, size_t ws_bytes,
                                    hipStream_t stream) {
  g_err.clear();
  mx_status st = validate_batch(batch, shape, nullptr);
  if (st != MX_OK) return st;
  if (req < 0 || req >= batch->num_reqs) return fail(MX_ERR_INVALID, "request %d out of range", req);
  if (!k_pool || !v_pool || !k_out || !v_out) return fail(MX_ERR_NULL, "tensor pointer is NULL");
  Plan p;
  build_plan(batch, shape, false, p);
  const Layout L = layout_for(p, shape, nullptr);
  if ((st = check_ws(L, ws, ws_bytes)) != MX_OK) return st;
  if ((st = upload_meta(p, L, shape, 1e4f, ws, stream)) != MX_OK) return st;
  const ReqDev& rq = p.reqs[req];
  hipError_t e = launch_gather(k_pool, v_pool, at<int32_t>(ws, L.pages) + rq.page_start, rq.kv_len,
                               shape->n_kv_heads, shape->head_dim, k_out, v_out, stream);
  if (e != hipSuccess) return hip_fail(e, "gather launch");
  return MX_OK;
}

MX_EXPORT size_t mx_debug_gemm_ws_bytes(int32_t M, int32_t N, int32_t K) {
  if (M < 0 || N <= 0 || K <= 0) return 0;
  return align_up(gemm_scratch_floats(M, N, K) * 4 + 4);
}

MX_EXPORT mx_status mx_debug_gemm(int32_t M, int32_t N, int32_t K, const uint16_t* A,
                                  const uint16_t* B, uint16_t* C, const uint16_t* R,
                                  int32_t epilogue, void* ws, size_t ws_bytes, hipStream_t stream) {
  return mx_debug_gemm_config(M, N, K, A, B, C, R, epilogue, -1, 0, ws, ws_bytes, stream);
}

namespace {
mx_status debug_gemm(int32_t M, int32_t N, int32_t K, const uint16_t* A, const uint16_t* B,
                     bool b_tiled, uint16_t* C, const uint16_t* R, int32_t epilogue,
                     int32_t tile_cfg, int32_t ksplit, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
  g_err.clear();
  if (b_tiled && (N % 16 || K % 32))
    return fail(MX_ERR_UNSUPPORTED, "tiled weights need N %% 16 == 0 and K %% 32 == 0");
  if (M < 0 || N <= 0 || K <= 0) return fail(MX_ERR_INVALID, "bad GEMM shape %d x %d x %d", M, N, K);
  if (K % 64) return fail(MX_ERR_UNSUPPORTED, "K %d is not a multiple of 64", K);
  if (tile_cfg < -1 || tile_cfg >= gemm_num_configs())
    return fail(MX_ERR_INVALID, "tile config %d out of range", tile_cfg);
  if (tile_cfg >= 0 && (ksplit < 1 || ksplit > 64 || K / 64 < ksplit))
    return fail(MX_ERR_INVALID, "K split %d is not in [1, min(64, K / 64 = %d)]", ksplit, K / 64);
  if (epilogue < 0 || epilogue > 2) return fail(MX_ERR_INVALID, "bad epilogue %d", epilogue);
  if (epilogue == EPI_SWIGLU && N % 64) return fail(MX_ERR_UNSUPPORTED, "SwiGLU needs N % 64 == 0");
  if (M == 0) return MX_OK;
  if (!A || !B || !C || (epilogue == EPI_RESIDUAL && !R)) return fail(MX_ERR_NULL, "NULL operand");
  if (mx_status sa = check_aligned({A, B, C, R, ws}); sa != MX_OK) return sa;
  if (epilogue == EPI_RESIDUAL) {
    const size_t bytes = (size_t)M * N * 2;  // C and R are both [M][N]
    const char *c0 = (const char*)C, *r0 = (const char*)R;
    if (c0 < r0 + bytes && r0 < c0 + bytes) return fail(MX_ERR_INVALID, "R overlaps C");
  }
  const size_t need = tile_cfg >= 0 ? (ksplit > 1 ? (size_t)ksplit * M * N : 0)
                                    : gemm_scratch_floats(M, N, K);
  if (need && (!ws || ws_bytes < need * 4))
    return fail(MX_ERR_TOO_LARGE, "GEMM scratch %zu bytes < %zu", ws_bytes, need * 4);
  DeviceState* ds;
  mx_status st = device_state(&ds);
  if (st != MX_OK) return st;
  const int ldc = epilogue == EPI_SWIGLU ? N / 2 : N;
  GemmArgs g{A, B, C, R, (float*)ws, M, N, K, K, K, ldc, N, epilogue, {}};
  if (b_tiled) {  // the layer step's operand layouts
    set_b_tiled(g);
    g.a_tiled = 1;
    g.c_tiled = epilogue == EPI_SWIGLU;
  } else {
    set_b_row_major(g);
  }
  hipError_t e = launch_gemm_config(g, ws ? ws_bytes / 4 : 0, tile_cfg, ksplit, stream);
  if (e != hipSuccess) return hip_fail(e, "gemm launch");
  return MX_OK;
}
}  // namespace

MX_EXPORT mx_status mx_debug_gemm_config(int32_t M, int32_t N, int32_t K, const uint16_t* A,
                                         const uint16_t* B, uint16_t* C, const uint16_t* R,
                                         int32_t epilogue, int32_t tile_cfg, int32_t ksplit,
                                         void* ws, size_t ws_bytes, hipStream_t stream) {
  return debug_gemm(M, N, K, A, B, false, C, R, epilogue, tile_cfg, ksplit, ws, ws_bytes, stream);
}

MX_EXPORT mx_status mx_debug_gemm_tiled(int32_t M, int32_t N, int32_t K, const uint16_t* A,
                                        const uint16_t* B_tiled, uint16_t* C, const uint16_t* R,
                                        int32_t epilogue, int32_t tile_cfg, int32_t ksplit,
                                        void* ws, size_t ws_bytes, hipStream_t stream) {
  return debug_gemm(M, N, K, A, B_tiled, true, C, R, epilogue, tile_cfg, ksplit, ws, ws_bytes,
                    stream);
}

MX_EXPORT mx_status mx_debug_gemm_plan(int32_t M, int32_t N, int32_t K, int32_t plan[5]) {
  g_err.clear();
  if (M < 0 || N <= 0 || K <= 0 || K % 64) return fail(MX_ERR_INVALID, "bad GEMM shape %d x %d x %d", M, N, K);
  if (!plan) return fail(MX_ERR_NULL, "plan is NULL");
  int out[5];
  gemm_plan(M, N, K, out);
  for (int i = 0; i < 5; i++) plan[i] = out[i];
  return MX_OK;
}

MX_EXPORT mx_status mx_debug_gemm_rows(int32_t M, int32_t N, int32_t K, const uint16_t* A,
                                       const uint16_t* B_tiled, uint16_t* C, const uint16_t* R,
                                       int32_t epilogue, int32_t m_main, int32_t main_cfg,
                                       int32_t tail_cfg, int32_t tail_ksplit, void* ws,
                                       size_t ws_bytes, hipStream_t stream) {
  g_err.clear();
  if (M < 2 || N <= 0 || K <= 0) return fail(MX_ERR_INVALID, "bad GEMM shape %d x %d x %d", M, N, K);
  if (N % 16 || K % 64) return fail(MX_ERR_UNSUPPORTED, "tiled weights need N %% 16 == 0 and K %% 64 == 0");
  if (m_main < 1 || m_main >= M || m_main % 16)
    return fail(MX_ERR_INVALID, "m_main %d not a multiple of 16 in [1, M)", m_main);
  if (main_cfg < 0 || main_cfg >= gemm_num_configs() || tail_cfg < 0 || tail_cfg >= gemm_num_configs())
    return fail(MX_ERR_INVALID, "tile config out of range");
  if (tail_ksplit < 1 || tail_ksplit > 64 || K / 64 < tail_ksplit)
    return fail(MX_ERR_INVALID, "K split %d is not in [1, min(64, K / 64 = %d)]", tail_ksplit, K / 64);
  if (epilogue < 0 || epilogue > 2) return fail(MX_ERR_INVALID, "bad epilogue %d", epilogue);
  if (epilogue == EPI_SWIGLU && N % 64) return fail(MX_ERR_UNSUPPORTED, "SwiGLU needs N % 64 == 0");
  if (!A || !B_tiled || !C || (epilogue == EPI_RESIDUAL && !R)) return fail(MX_ERR_NULL, "NULL operand");
  if (mx_status sa = check_aligned({A, B_tiled, C, R, ws}); sa != MX_OK) return sa;
  if (epilogue == EPI_RESIDUAL) {
    const size_t bytes = (size_t)M * N * 2;
    const char *c0 = (const char*)C, *r0 = (const char*)R;
    if (c0 < r0 + bytes && r0 < c0 + bytes) return fail(MX_ERR_INVALID, "R overlaps C");
  }
  const size_t need = tail_ksplit > 1 ? (size_t)tail_ksplit * (M - m_main) * N : 0;
  if (need && (!ws || ws_bytes < need * 4))
    return fail(MX_ERR_TOO_LARGE, "GEMM scratch %zu bytes < %zu", ws_bytes, need * 4);
  DeviceState* ds;
  mx_status st = device_state(&ds);
  if (st != MX_OK) return st;
  const int ldc = epilogue == EPI_SWIGLU ? N / 2 : N;
  GemmArgs g{A, B_tiled, C, R, (float*)ws, M, N, K, K, K, ldc, N, epilogue, {}};
  set_b_tiled(g);
  g.a_tiled = 1;
  g.c_tiled = epilogue == EPI_SWIGLU;
  hipError_t e = launch_gemm_rows(g, ws ? ws_bytes / 4 : 0, m_main, main_cfg, tail_cfg, tail_ksplit,
                                  stream);
  if (e != hipSuccess) return hip_fail(e, "gemm launch");
  return MX_OK;
}

MX_EXPORT mx_status mx_debug_reduce_residual_rmsnorm(const float* partial, int32_t ksplit,
                                                     const uint16_t* R, uint16_t* x1,
                                                     const uint16_t* g, uint16_t* h, int32_t M,
                                                     int32_t H, float eps, int32_t split_row,
                                                     hipStream_t stream) {
  g_err.clear();
  if (M < 0 || H <= 0 || H % 32) return fail(MX_ERR_INVALID, "bad shape %d x %d", M, H);
  if (H > kFusedNormMaxH) return fail(MX_ERR_UNSUPPORTED, "H %d > %d", H, kFusedNormMaxH);
  if (ksplit < 1) return fail(MX_ERR_INVALID, "ksplit %d < 1", ksplit);
  if (split_row < 0 || split_row > M) return fail(MX_ERR_INVALID, "split_row %d not in [0, M]", split_row);
  if (M == 0) return MX_OK;
  if ((split_row < M && !partial) || !R || !x1 || !g || !h) return fail(MX_ERR_NULL, "NULL operand");
  if (mx_status sa = check_aligned({partial, R, x1, g, h}); sa != MX_OK) return sa;
  DeviceState* ds;
  mx_status st = device_state(&ds);
  if (st != MX_OK) return st;
  hipError_t e = launch_reduce_residual_rmsnorm(partial, ksplit, R, x1, g, h, M, H, eps, split_row,
                                                stream);
  if (e != hipSuccess) return hip_fail(e, "reduce launch");
  return MX_OK;
}

MX_EXPORT mx_status mx_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> g(g_prof.mu);
  g_prof.on = on != 0;
  return MX_OK;
}

MX_EXPORT int32_t mx_profile_read(const char** names, float* total_ms, int32_t* counts,
                                  int32_t max_entries) {
  std::lock_guard<std::mutex> g(g_prof.mu);
  for (auto& r : g_prof.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      size_t i = 0;
      while (i < g_prof.names.size() && strcmp(g_prof.names[i], r.name) != 0) i++;
      if (i == g_prof.names.size()) {
        g_prof.names.push_back(r.name);
        g_prof.total_ms.push_back(0.0);
        g_prof.counts.push_back(0);
      }
      g_prof.total_ms[i] += ms;
      g_prof.counts[i] += 1;
    }
    g_prof.free_events.push_back(r.a);
    g_prof.free_events.push_back(r.b);
  }
  g_prof.pending.clear();
  const int32_t n = (int32_t)std::min<size_t>(g_prof.names.size(), (size_t)std::max(0, max_entries));
  for (int32_t i = 0; i < n; i++) {
    if (names) names[i] = g_prof.names[i];
    if (total_ms) total_ms[i] = (float)g_prof.total_ms[i];
    if (counts) counts[i] = g_prof.counts[i];
  }
  g_prof.names.clear();
  g_prof.total_ms.clear();
  g_prof.counts.clear();
  return n;
}
