// C ABI of the link-stage attention library: the chunk store (pool +
// hash table + bump allocator), the per-call link planner and its staging of
// the chunk table, kernel selection, and kernel timing.
#include "../../include/pic.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <map>
#include <initializer_list>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "pic_internal.hpp"

namespace pic {
size_t valu_lds_bytes_for(int esz, int mla, int d_k, int d_v);
}

using namespace pic;

namespace {

thread_local std::string g_err;

pic_status fail(pic_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

pic_status hip_fail(hipError_t e, const char *what) {
  return fail(PIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                 \
  do {                                      \
    hipError_t e_ = (expr);                 \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = true, switched = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) { ok = false; return; }
    if (prev != dev) {
      switched = true;
      if (hipSetDevice(dev) != hipSuccess) ok = false;
    }
  }
  ~DeviceGuard() {
    if (switched && prev >= 0) (void)hipSetDevice(prev);
  }
};

// The pool is a sequence of 64-token pages (one attention tile each). A
// chunk occupies runs of consecutive pages -- one run whenever a free run
// is long enough -- and each run holds a piece of the chunk laid out like a
// chunk of its own (K [H][run tokens][d_k], then V^T [H][d_v][run tokens]),
// so a piece is one link-table entry and the kernels need no page table.
// Such a run of pages is a block; a chunk is a list of views of blocks
// (pages skip .. of the block), in token order. A chunk made by
// pic_store_derive views its base's blocks for the pages it shares with
// it, so blocks are reference-counted by the chunks that view them.
struct Run {
  int64_t page0;        // the block's first page
  int32_t pages;        // the block's pages (its row stride is pages * 64 tokens)
  int32_t tok0;         // first chunk token held by the view
  int32_t ntok;         // chunk tokens held by the view
  int32_t skip = 0;     // pages of the block before the view's first page
};

struct Slot {
  int64_t len;
  std::vector<Run> runs;
  int64_t plan_refs = 0;   // live link plans that link this chunk
  bool derived = false;    // made by pic_store_derive (rows may be written)
};

// Pinned host table + device copy + completion event. The planner writes a
// call's chunk/request tables into one slot, copies them to the device on
// the call's stream, and records the event after the call's last kernel; a
// slot is reused only after its event has completed.
// A call's workspace (own-KV slots, split partials) belongs to its slot
// too, so calls in flight on different streams never share one.
struct Stage {
  void *host = nullptr;
  void *host_dev = nullptr;     // device-visible address of host
  void *dev = nullptr;
  size_t cap = 0;
  void *work = nullptr;
  size_t work_cap = 0;
  hipEvent_t done = nullptr;
  bool pending = false;
};

constexpr int kRing = 8;

struct ProfState {
  std::mutex mu;
  bool on = false;
  int32_t every = 1;       // time one launch in `every`
  int64_t seen = 0;        // launches since the last begin
  std::vector<std::pair<hipEvent_t, hipEvent_t>> events;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> spare;
  std::string name;
};
ProfState g_prof;

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

}  // namespace

namespace pic {
// Queried once per device: compute units, and XCDs (one when the runtime
// does not report them, e.g. a partition that exposes a single die).
DevShape device_shape() {
  static std::mutex mu;
  static std::unordered_map<int, DevShape> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DevShape{256, 8};
  std::lock_guard<std::mutex> g(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) return it->second;
  int cus = 0, xcds = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    cus = 256;
  if (hipDeviceGetAttribute(&xcds, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || xcds <= 0)
    xcds = 1;
  (void)hipGetLastError();
  const DevShape ds{cus, xcds};
  cache.emplace(dev, ds);
  return ds;
}
}  // namespace pic

struct pic_store {
  pic_store_desc desc{};
  int device = 0;
  int esz = 2;
  char *pool = nullptr;
  int64_t capacity = 0;          // padded tokens
  int64_t used = 0;              // tokens of allocated pages
  std::map<int64_t, int64_t> free_runs;   // page0 -> pages, coalesced
  std::unordered_map<int64_t, int32_t> block_refs;   // block page0 -> chunks viewing it
  std::vector<int32_t> page_refs;                     // page -> chunks viewing it
  // runs of removed chunks, reusable once the event (recorded on the
  // remover's stream) has completed
  std::vector<std::pair<hipEvent_t, std::vector<Run>>> pending;
  int32_t n_layers = 1;
  int64_t layer_bytes = 0;       // bytes of one layer's pool; layer l of a slot is l * layer_bytes on
  int64_t live_plans = 0;
  int64_t k_tok_elems = 0;       // K elements per padded token (all heads)
  int64_t v_tok_elems = 0;       // V elements per padded token (GQA)
  std::unordered_map<uint64_t, Slot> map;
  Stage ring[kRing];
  int next = 0;
  DevShape shape{256, 8};        // compute units and XCDs of the store's device
  bool imported = false;         // pool mapped from another process (read-only)
  // request order of the last multi-round d128 prefill call and its key
  // (the request shapes; see balance_order_d128)
  std::vector<int32_t> order_key, order_memo;
};

namespace {

pic_status stage_acquire(pic_store *s, size_t bytes, Stage **out) {
  Stage &st = s->ring[s->next];
  s->next = (s->next + 1) % kRing;
  if (st.pending) {
    HIP_TRY(hipEventSynchronize(st.done), "hipEventSynchronize(stage)");
    st.pending = false;
  }
  // Completion only (the host waits for the copy out of the staging buffer
  // to be done): no system-scope fence, which would write back and
  // invalidate caches after every call.
  if (!st.done)
    HIP_TRY(hipEventCreateWithFlags(&st.done, hipEventDisableTiming | hipEventDisableSystemFence),
            "hipEventCreate");
  if (st.cap < bytes) {
    if (st.host) (void)hipHostFree(st.host);
    if (st.dev) (void)hipFree(st.dev);
    st.host = st.dev = nullptr;
    st.cap = 0;
    size_t cap = std::max<size_t>(round_up((int64_t)bytes, 4096), 64 * 1024);
    HIP_TRY(hipHostMalloc(&st.host, cap, hipHostMallocDefault), "hipHostMalloc(stage)");
    HIP_TRY(hipHostGetDevicePointer(&st.host_dev, st.host, 0), "hipHostGetDevicePointer(stage)");
    HIP_TRY(hipMalloc(&st.dev, cap), "hipMalloc(stage)");
    st.cap = cap;
  }
  *out = &st;
  return PIC_OK;
}

// Grows the workspace of an acquired staging slot (whose previous call has
// completed, so the old buffer is free).
pic_status ensure_work(Stage *st, size_t bytes) {
  if (st->work_cap >= bytes) return PIC_OK;
  if (st->work) {
    (void)hipFree(st->work);
    st->work = nullptr;
    st->work_cap = 0;
  }
  size_t cap = round_up((int64_t)bytes, 1 << 20);
  HIP_TRY(hipMalloc(&st->work, cap), "hipMalloc(workspace)");
  st->work_cap = cap;
  return PIC_OK;
}

// Returns a run of pages to the free map, merging it with free neighbours.
void free_run(pic_store *s, int64_t page0, int64_t pages) {
  auto next = s->free_runs.lower_bound(page0);
  if (next != s->free_runs.end() && next->first == page0 + pages) {
    pages += next->second;
    next = s->free_runs.erase(next);
  }
  if (next != s->free_runs.begin()) {
    auto prev = std::prev(next);
    if (prev->first + prev->second == page0) {
      prev->second += pages;
      return;
    }
  }
  s->free_runs.emplace(page0, pages);
}

// Moves the runs of removed chunks whose readers have finished into the
// free map; with wait, first waits for all of them.
pic_status reclaim(pic_store *s, bool wait) {
  std::vector<std::pair<hipEvent_t, std::vector<Run>>> keep;
  for (auto &pr : s->pending) {
    hipError_t e = wait ? hipEventSynchronize(pr.first) : hipEventQuery(pr.first);
    if (e == hipErrorNotReady) {
      keep.push_back(std::move(pr));
      continue;
    }
    if (e != hipSuccess) return hip_fail(e, "removed-chunk event");
    (void)hipEventDestroy(pr.first);
    for (const Run &r : pr.second) {
      free_run(s, r.page0, r.pages);
      s->used -= (int64_t)r.pages * kTile;
    }
  }
  s->pending.swap(keep);
  return PIC_OK;
}

// Allocates `pages` pages: the first free run that is long enough, else the
// longest free runs until the request is met. false if the pool is short.
bool alloc_pages(pic_store *s, int64_t pages, std::vector<Run> &out) {
  out.clear();
  for (auto it = s->free_runs.begin(); it != s->free_runs.end(); ++it) {
    if (it->second < pages) continue;
    out.push_back(Run{it->first, (int32_t)pages, 0, 0});
    const int64_t rest = it->second - pages, start = it->first + pages;
    s->free_runs.erase(it);
    if (rest > 0) s->free_runs.emplace(start, rest);
    return true;
  }
  int64_t total = 0;
  for (auto &fr : s->free_runs) total += fr.second;
  if (total < pages) return false;
  std::vector<std::pair<int64_t, int64_t>> runs(s->free_runs.begin(), s->free_runs.end());
  std::stable_sort(runs.begin(), runs.end(),
                   [](const std::pair<int64_t, int64_t> &a, const std::pair<int64_t, int64_t> &b) {
                     return a.second > b.second;
                   });
  int64_t need = pages;
  for (auto &r : runs) {
    const int64_t take = std::min(need, r.second);
    out.push_back(Run{r.first, (int32_t)take, 0, 0});
    s->free_runs.erase(r.first);
    if (take < r.second) s->free_runs.emplace(r.first + take, r.second - take);
    need -= take;
    if (need == 0) break;
  }
  std::sort(out.begin(), out.end(), [](const Run &a, const Run &b) { return a.page0 < b.page0; });
  return true;
}

// Link-table entry of one run of a chunk in `layer`.
LinkEntry run_entry(const pic_store *s, const Run &r, int32_t layer) {
  const int64_t slot_tok_bytes = (s->k_tok_elems + s->v_tok_elems) * s->esz;
  const int32_t lp = r.pages * kTile;
  const int64_t skip_tok = (int64_t)r.skip * kTile;
  const char *block = s->pool + (int64_t)layer * s->layer_bytes + r.page0 * kTile * slot_tok_bytes;
  LinkEntry E{};
  // K rows and V^T panels of the view start skip_tok tokens into the block
  // (skip_tok is a multiple of the 32-token panel: skip_tok * d_v elements)
  E.k = block + skip_tok * s->desc.d_k * s->esz;
  E.v = s->desc.kind == PIC_GQA
            ? block + (int64_t)lp * s->k_tok_elems * s->esz + skip_tok * s->desc.d_v * s->esz
            : E.k;
  E.len = r.ntok;
  E.lp = lp;
  return E;
}

// Pages for a new chunk: free ones, else those of removed chunks whose
// readers are done, else after waiting for the remaining readers.
pic_status take_pages(pic_store *s, int64_t pages, std::vector<Run> &runs) {
  runs.clear();
  if (pages == 0) return PIC_OK;
  pic_status rc = reclaim(s, false);
  if (rc != PIC_OK) return rc;
  if (!alloc_pages(s, pages, runs) && !s->pending.empty()) {
    rc = reclaim(s, true);
    if (rc != PIC_OK) return rc;
    (void)alloc_pages(s, pages, runs);
  }
  if (runs.empty())
    return fail(PIC_ERR_OOM, "pool full: %lld of %lld tokens in use, %lld needed",
                (long long)s->used, (long long)s->capacity, (long long)pages * kTile);
  return PIC_OK;
}

// Host row list of pic_store_derive / pic_store_write_rows: strictly
// increasing, each below len.
bool check_rows(const int32_t *rows, int32_t n, int64_t len) {
  if (n < 0 || (n > 0 && !rows)) return false;
  for (int32_t i = 0; i < n; ++i)
    if (rows[i] < 0 || rows[i] >= len || (i > 0 && rows[i] <= rows[i - 1])) return false;
  return true;
}

// Adds d to the reference count of every page a chunk's views cover.
void ref_pages(pic_store *s, const std::vector<Run> &views, int32_t d) {
  for (const Run &v : views) {
    const int64_t first = v.page0 + v.skip, n = (v.ntok + kTile - 1) / kTile;
    for (int64_t p = first; p < first + n; ++p) s->page_refs[p] += d;
  }
}

// The view of a chunk holding token t.
const Run &view_of(const Slot &sl, int64_t t) {
  size_t i = 0;
  while (i + 1 < sl.runs.size() && sl.runs[i].tok0 + sl.runs[i].ntok <= t) ++i;
  return sl.runs[i];
}

bool check_offsets(const int32_t *a, int32_t n) {
  if (!a || a[0] != 0) return false;
  for (int32_t i = 0; i < n; ++i)
    if (a[i + 1] < a[i]) return false;
  return true;
}

// Validated, resolved form of one link call.
struct Plan {
  std::vector<LinkEntry> links;  // per request: its document links, then its own KV
  std::vector<ReqEntry> reqs;
  std::vector<int32_t> order;
  std::vector<std::pair<int32_t, int64_t>> own;   // (link index, workspace byte offset)
  int64_t own_bytes = 0;
  int32_t max_own_lp = 0;
  int32_t total_q = 0;
  int32_t max_rows = 0;          // max over requests of lq * group
  int32_t max_tiles = 0;
  bool self = false;             // requests carry own KV
  int64_t total_self = 0;        // own tokens over the batch
  std::vector<uint64_t> ids;     // every linked chunk id (with repeats)
  // per query token: linked rows visible to it; empty unless the rows of
  // some request see different numbers of them (the kernels mask per row)
  std::vector<int32_t> doc_lim;
};

// Tensor arguments of a call against its plan.
pic_status check_tensors(const pic_store *s, const Plan &P, const void *q, const void *k_self,
                         const void *v_self, const void *out) {
  if (P.total_q > 0 && (!q || !out)) return fail(PIC_ERR_INVALID, "q/out is NULL");
  if (P.self) {
    if (P.total_self > 0 && !k_self) return fail(PIC_ERR_INVALID, "k_self is NULL");
    if (s->desc.kind == PIC_GQA && P.total_self > 0 && !v_self)
      return fail(PIC_ERR_INVALID, "v_self is NULL");
    if (s->desc.kind == PIC_MLA && v_self) return fail(PIC_ERR_INVALID, "v_self must be NULL for MLA");
  } else if (k_self || v_self) {
    return fail(PIC_ERR_INVALID, "k_self/v_self given without self_offsets");
  }
  return PIC_OK;
}

// Validates a request batch and resolves its chunk ids into the link and
// request tables, with chunk addresses in cross-attention layer `layer`.
pic_status plan_call(pic_store *s, const pic_link_req *req, int32_t n_q_heads, float scale,
                     int32_t layer, int32_t max_q_per_req, Plan &P) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (!req) return fail(PIC_ERR_INVALID, "req is NULL");
  if (layer < 0 || layer >= s->n_layers)
    return fail(PIC_ERR_INVALID, "layer %d outside the store's %d layers", layer, s->n_layers);
  const pic_store_desc &d = s->desc;
  const int32_t B = req->batch;
  if (B < 0) return fail(PIC_ERR_INVALID, "batch < 0");
  if (n_q_heads <= 0 || n_q_heads % d.n_kv_heads)
    return fail(PIC_ERR_INVALID, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
                n_q_heads, d.n_kv_heads);
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(PIC_ERR_INVALID, "softmax_scale must be positive and finite");
  if (B == 0) return PIC_OK;
  if (!check_offsets(req->chunk_offsets, B)) return fail(PIC_ERR_INVALID, "bad chunk_offsets");
  if (!check_offsets(req->q_offsets, B)) return fail(PIC_ERR_INVALID, "bad q_offsets");
  const bool self = req->self_offsets != nullptr;
  if (self && !check_offsets(req->self_offsets, B)) return fail(PIC_ERR_INVALID, "bad self_offsets");
  const int64_t n_links = req->chunk_offsets[B];
  const int64_t tq = req->q_offsets[B];
  const int64_t ts = self ? req->self_offsets[B] : 0;
  if (n_links > 0 && !req->chunk_ids) return fail(PIC_ERR_INVALID, "chunk_ids is NULL");
  if (tq * n_q_heads > INT32_MAX / 2) return fail(PIC_ERR_INVALID, "too many query rows");
  P.self = self;
  P.total_self = ts;
  const int group = n_q_heads / d.n_kv_heads;
  const int64_t slot_tok_bytes = (s->k_tok_elems + s->v_tok_elems) * s->esz;
  P.links.clear();
  P.links.reserve(n_links + B);
  P.ids.clear();
  P.reqs.resize(B);
  P.doc_lim.clear();
  bool mixed_limits = false;
  std::vector<int64_t> weight(B);
  for (int32_t r = 0; r < B; ++r) {
    ReqEntry &R = P.reqs[r];
    const int32_t c0 = req->chunk_offsets[r], nc = req->chunk_offsets[r + 1] - c0;
    R.link0 = (int32_t)P.links.size();
    R.q0 = req->q_offsets[r];
    R.lq = req->q_offsets[r + 1] - R.q0;
    R.s0 = self ? req->self_offsets[r] : 0;
    R.ls = self ? req->self_offsets[r + 1] - R.s0 : 0;
    if (self && R.ls < R.lq)
      return fail(PIC_ERR_INVALID, "request %d: %d query tokens but only %d own tokens", r, R.lq,
                  R.ls);
    if (R.lq > max_q_per_req)
      return fail(PIC_ERR_INVALID, "request %d: %d query tokens exceeds %d", r, R.lq,
                  max_q_per_req);
    int64_t tiles = 0, toks = 0;
    for (int32_t c = 0; c < nc; ++c) {
      const uint64_t id = req->chunk_ids[c0 + c];
      auto it = s->map.find(id);
      if (it == s->map.end())
        return fail(PIC_ERR_NOT_FOUND, "request %d link %d: chunk id 0x%llx not in the store", r,
                    c, (unsigned long long)id);
      const Slot &sl = it->second;
      const int32_t start = req->chunk_starts ? req->chunk_starts[c0 + c] : 0;
      if (start < 0 || start % kTile || start >= sl.len)
        return fail(PIC_ERR_INVALID,
                    "request %d link %d: start %d must be a multiple of %d below the chunk's %lld "
                    "tokens", r, c, start, kTile, (long long)sl.len);
      for (const Run &run : sl.runs) {
        if (run.tok0 + run.ntok <= start) continue;
        LinkEntry E = run_entry(s, run, layer);
        // skip the run's pages before `start`: rows of K, panels of V^T
        // (the head stride stays the run's)
        const int32_t skip = std::max(0, start - run.tok0);
        E.k = (const char *)E.k + (int64_t)skip * d.d_k * s->esz;
        E.v = d.kind == PIC_MLA ? E.k : (const char *)E.v + (int64_t)skip * d.d_v * s->esz;
        E.len -= skip;
        E.tile0 = (int32_t)tiles;
        E.tok0 = (int32_t)toks;
        P.links.push_back(E);
        tiles += (E.len + kTile - 1) / kTile;
        toks += E.len;
      }
      P.ids.push_back(id);
    }
    if (req->q_doc_limits && R.lq > 0) {
      int32_t lo = INT32_MAX, hi = 0;
      for (int32_t i = 0; i < R.lq; ++i) {
        const int32_t lim = req->q_doc_limits[R.q0 + i];
        if (lim < 0 || lim > toks)
          return fail(PIC_ERR_INVALID, "request %d query %d: limit %d outside 0..%lld linked rows",
                      r, i, lim, (long long)toks);
        lo = std::min(lo, lim);
        hi = std::max(hi, lim);
      }
      // rows past every query's limit are never read: cut the links there;
      // limits that differ between rows are applied by the kernels
      if (hi < toks) {
        size_t keep = R.link0;
        tiles = 0;
        while (keep < P.links.size() && P.links[keep].tok0 < hi) {
          LinkEntry &E = P.links[keep++];
          E.len = std::min(E.len, hi - E.tok0);
          tiles += (E.len + kTile - 1) / kTile;
        }
        P.links.resize(keep);
        toks = hi;
      }
      if (lo < hi) mixed_limits = true;
    }
    if (toks + R.ls > INT32_MAX / 2) return fail(PIC_ERR_INVALID, "request %d too long", r);
    R.doc_tiles = (int32_t)tiles;
    if (R.ls > 0) {             // own KV: a slot in the call's workspace, filled on the device
      LinkEntry E{};
      E.len = R.ls;
      E.lp = (int32_t)round_up(R.ls, kTile);
      E.tile0 = (int32_t)tiles;
      E.tok0 = (int32_t)toks;
      P.own.emplace_back((int32_t)P.links.size(), P.own_bytes);
      P.own_bytes += round_up((int64_t)E.lp * slot_tok_bytes, 256);
      P.max_own_lp = std::max(P.max_own_lp, E.lp);
      P.links.push_back(E);
      tiles += E.lp / kTile;
    }
    R.nlinks = (int32_t)P.links.size() - R.link0;
    R.tiles = (int32_t)tiles;
    P.max_rows = std::max(P.max_rows, R.lq * group);
    P.max_tiles = std::max(P.max_tiles, R.tiles);
    weight[r] = (int64_t)R.tiles * R.lq;
  }
  P.order.resize(B);
  for (int32_t r = 0; r < B; ++r) P.order[r] = r;
  std::stable_sort(P.order.begin(), P.order.end(),
                   [&](int32_t a, int32_t b) { return weight[a] > weight[b]; });
  P.total_q = (int32_t)tq;
  if (mixed_limits) P.doc_lim.assign(req->q_doc_limits, req->q_doc_limits + tq);
  return PIC_OK;
}

// Points the own-KV links of `links` (the plan's tables) at their slots in
// the workspace `work`.
void place_own(const pic_store *s, const Plan &P, void *work, LinkEntry *links) {
  const bool mla = s->desc.kind == PIC_MLA;
  for (auto &o : P.own) {
    LinkEntry &E = links[o.first];
    E.k = (char *)work + o.second;
    E.v = mla ? E.k : (const char *)E.k + (int64_t)E.lp * s->k_tok_elems * s->esz;
  }
}

// Writes the plan's tables into a staging slot (host-mapped pinned memory)
// and points lp's tables at the slot's device copy; the call's prologue
// kernel moves them there.
struct TableLayout {
  size_t off_r, off_o, off_d, bytes;
};

// Where the prologue reads the tables, and what it copies first.
struct Prologue {
  const LinkEntry *links = nullptr;
  const ReqEntry *reqs = nullptr;
  const void *copy_src = nullptr;
  void *copy_dst = nullptr;
  int64_t copy_bytes = 0;
};

// The slot also holds the call's workspace (work_bytes), where the own-KV
// links are pointed.
pic_status upload(pic_store *s, Plan &P, size_t work_bytes, Stage **stage, LinkParams &lp,
                  TableLayout &tl) {
  const size_t nl = P.links.size(), nr = P.reqs.size();
  tl.off_r = round_up(sizeof(LinkEntry) * nl, 256);
  tl.off_o = tl.off_r + round_up(sizeof(ReqEntry) * nr, 256);
  tl.off_d = tl.off_o + round_up(sizeof(int32_t) * nr, 256);
  tl.bytes = tl.off_d + round_up(sizeof(int32_t) * P.doc_lim.size(), 256);
  const size_t off_r = tl.off_r, off_o = tl.off_o, bytes = tl.bytes;
  pic_status rc = stage_acquire(s, bytes, stage);
  if (rc != PIC_OK) return rc;
  if (work_bytes > 0) {
    rc = ensure_work(*stage, work_bytes);
    if (rc != PIC_OK) return rc;
  }
  place_own(s, P, (*stage)->work, P.links.data());
  char *h = (char *)(*stage)->host;
  if (nl) memcpy(h, P.links.data(), sizeof(LinkEntry) * nl);
  memcpy(h + off_r, P.reqs.data(), sizeof(ReqEntry) * nr);
  memcpy(h + off_o, P.order.data(), sizeof(int32_t) * nr);
  if (!P.doc_lim.empty()) memcpy(h + tl.off_d, P.doc_lim.data(), sizeof(int32_t) * P.doc_lim.size());
  char *dv = (char *)(*stage)->dev;
  lp.links = (const LinkEntry *)dv;
  lp.reqs = (const ReqEntry *)(dv + off_r);
  lp.order = (const int32_t *)(dv + off_o);
  lp.doc_lim = P.doc_lim.empty() ? nullptr : (const int32_t *)(dv + tl.off_d);
  return PIC_OK;
}

void prof_start(hipStream_t st, std::pair<hipEvent_t, hipEvent_t> *ev) {
  ev->first = ev->second = nullptr;
  std::lock_guard<std::mutex> g(g_prof.mu);
  if (!g_prof.on) return;
  if (g_prof.seen++ % g_prof.every) return;
  if (!g_prof.spare.empty()) {
    *ev = g_prof.spare.back();
    g_prof.spare.pop_back();
  } else if (hipEventCreateWithFlags(&ev->first, hipEventDisableSystemFence) != hipSuccess ||
             hipEventCreateWithFlags(&ev->second, hipEventDisableSystemFence) != hipSuccess) {
    // timing-only events: a system-scope fence would add a cache writeback
    // and invalidation around the timed kernel
    ev->first = ev->second = nullptr;
    return;
  }
  (void)hipEventRecord(ev->first, st);
}

void prof_stop(hipStream_t st, std::pair<hipEvent_t, hipEvent_t> *ev, const char *name) {
  if (!ev->first) return;
  (void)hipEventRecord(ev->second, st);
  std::lock_guard<std::mutex> g(g_prof.mu);
  g_prof.events.push_back(*ev);
  g_prof.name = name;
}

enum class Mode { Prefill, Decode };
enum class Kern { Valu, Mfma128, Decode128, Mla };

// Everything about a call that does not depend on its tensors: the resolved
// tables, the kernel, the split count and the workspace layout
// [own KV slots, laid out like chunk slots][split partials].
struct Setup {
  Plan P;
  Kern kern = Kern::Valu;
  int32_t splits = 1;
  bool lean = false;             // a small call the lean kernel runs
  LinkParams lp{};               // shapes only: no tables, tensors or scale yet
  std::vector<OwnArg> own_args;  // per request, for the prologue (batch <= kOwnArgs)
  size_t part_off = 0, part_bytes = 0;
  size_t work_bytes() const { return part_off + part_bytes; }
};

// Request order for the d128 prefill kernel. Workgroup j of XCD x runs row
// block j % nrb of group x + n_xcd (j / nrb) (see the kernel's work
// mapping) and starts on the first of the XCD's slots (CUs times workgroups
// per CU) that frees up, as the in-order dispatch does; with n_kv a multiple
// of n_xcd every XCD sees the same sequence of requests, each n_kv / n_xcd
// times. Heaviest first is the usual list-scheduling order; when an XCD's
// workgroups take several rounds of its slots, one pass of pairwise swaps
// that shorten the simulated finish time improves on it (long_rag: 957 ->
// 934 tiles, against a bound of 916). A workgroup takes its visible tiles
// plus 1.5 (its query rows, first tile and epilogue). The search keeps the
// slot times after each prefix of the order and stops a trial once some
// slot passes the best finish time; the result is kept for the next call
// with the same request shapes (a batch linked at every cross-attention
// layer or decode step). Other shapes keep heaviest first.
struct OrderSim {
  const Plan *P;
  int nrb, rows_per_block, group, reps, slots;
  double dur(int r, int rb) const {
    const ReqEntry &R = P->reqs[r];
    const int rows = R.lq * group, row0 = rb * rows_per_block;
    if (row0 >= rows) return -1.0;    // the workgroup returns at once
    return visible_tiles(R, std::min(rows - 1, row0 + rows_per_block - 1) / group) + 1.5;
  }
  // Adds request r's workgroups to the slot times `h` (a min-heap); false
  // once some slot passes `limit`.
  bool add(std::vector<double> &h, double &top, int r, double limit) const {
    for (int k = 0; k < reps; ++k)
      for (int rb = 0; rb < nrb; ++rb) {
        const double d = dur(r, rb);
        if (d < 0) continue;
        std::pop_heap(h.begin(), h.end(), std::greater<double>());
        h.back() += d;
        top = std::max(top, h.back());
        std::push_heap(h.begin(), h.end(), std::greater<double>());
        if (top >= limit) return false;
      }
    return true;
  }
};

// finish: when not NULL, receives the simulated finish time (in tiles) of
// the busiest XCD for heaviest first and for the order chosen (both 0 when
// no search runs). s: the store whose memo to use, or NULL for none.
void balance_order_d128(pic_store *s, Plan &P, const LinkParams &lp, int rows_per_block,
                        int slots, double *finish = nullptr) {
  if (finish) finish[0] = finish[1] = 0;
  const int B = (int)P.order.size();
  if (B < 3 || B > 64 || slots <= 0 || lp.n_kv_heads % lp.n_xcd) return;
  const int reps = lp.n_kv_heads / lp.n_xcd;
  if ((int64_t)B * reps * lp.nrb <= slots) return;   // one round: all start at once
  std::vector<int32_t> key = {lp.nrb, rows_per_block, lp.group, reps, slots, B};
  for (const ReqEntry &R : P.reqs) key.insert(key.end(), {R.lq, R.ls, R.doc_tiles, R.tiles});
  if (s && !finish && key == s->order_key) {
    P.order = s->order_memo;
    return;
  }
  const OrderSim sim{&P, lp.nrb, rows_per_block, lp.group, reps, slots};
  std::vector<int32_t> order = P.order;
  std::vector<double> pre(slots, 0.0), h;
  double pre_top = 0, best = 0;
  {
    h = pre;
    for (int i = 0; i < B; ++i) sim.add(h, best, order[i], INFINITY);
  }
  if (finish) finish[0] = best;
  auto same_shape = [&](int a, int b) {
    const ReqEntry &x = P.reqs[a], &y = P.reqs[b];
    return x.lq == y.lq && x.ls == y.ls && x.doc_tiles == y.doc_tiles && x.tiles == y.tiles;
  };
  for (int i = 0; i + 1 < B; ++i) {
    for (int j = i + 1; j < B; ++j) {
      if (same_shape(order[i], order[j])) continue;
      std::swap(order[i], order[j]);
      h = pre;
      double top = pre_top;
      bool ok = true;
      for (int k = i; k < B && ok; ++k) ok = sim.add(h, top, order[k], best - 1e-9);
      if (ok)
        best = top;
      else
        std::swap(order[i], order[j]);
    }
    sim.add(pre, pre_top, order[i], INFINITY);
  }
  if (finish) finish[1] = best;
  P.order = order;
  if (s) {
    s->order_key = std::move(key);
    s->order_memo = order;
  }
}

pic_status setup_call(pic_store *s, const pic_link_req *req, int32_t n_q_heads, float scale,
                      int32_t layer, int32_t num_splits, Mode mode, Setup &C) {
  if (mode == Mode::Decode && (num_splits < 0 || num_splits > 256))
    return fail(PIC_ERR_INVALID, "num_splits must be 0..256");
  Plan &P = C.P;
  pic_status rc = plan_call(s, req, n_q_heads, scale, layer,
                            mode == Mode::Decode ? 16 : INT32_MAX, P);
  if (rc != PIC_OK) return rc;
  const pic_store_desc &d = s->desc;
  const bool mla = d.kind == PIC_MLA;
  LinkParams &lp = C.lp;
  lp.batch = req->batch;
  lp.n_q_heads = n_q_heads;
  lp.n_kv_heads = d.n_kv_heads;
  lp.group = n_q_heads / d.n_kv_heads;
  lp.d_k = d.d_k;
  lp.d_v = d.d_v;
  lp.total_q = P.total_q;
  if (req->batch == 0 || P.total_q == 0) return PIC_OK;
  if (P.max_own_lp > 0 && req->batch <= kOwnArgs) {
    C.own_args.assign(req->batch, OwnArg{0, 0, 0});
    size_t k = 0;
    for (int32_t r = 0; r < req->batch; ++r) {
      const ReqEntry &R = P.reqs[r];
      if (R.ls == 0) continue;
      C.own_args[r] = OwnArg{R.s0, R.ls, P.own[k++].second};
    }
  }

  // Kernel choice.
  //   bf16 GQA d=128: decode-shaped calls with at most 16 rows per (request,
  //   kv head) stream keys with the decode kernel; everything else runs the
  //   matrix-core flash kernel (split when decoding).
  //   Other shapes / fp32 / MLA: the generic vector-ALU kernel.
  //   bf16 MLA with 576-wide latent rows and 512-wide values: the MLA
  //   matrix-core kernel (split when decoding).
  Kern kern = Kern::Valu;
  const bool bf16_128 = d.dtype == PIC_BF16 && !mla && d.d_k == 128 && d.d_v == 128;
  if (bf16_128)
    kern = mode == Mode::Decode && P.max_rows <= decode_d128_max_rows() ? Kern::Decode128
                                                                         : Kern::Mfma128;
  // rows of one request that see different numbers of linked rows need the
  // per-row masks of the flash kernel
  if (kern == Kern::Decode128 && !P.doc_lim.empty()) kern = Kern::Mfma128;
  if (d.dtype == PIC_BF16 && mla && d.d_k == 576 && d.d_v == 512) kern = Kern::Mla;
  if (kern == Kern::Valu && valu_lds_bytes_for(s->esz, mla, d.d_k, d.d_v) > 160 * 1024)
    return fail(PIC_ERR_UNSUPPORTED, "head widths d_k=%d d_v=%d exceed the generic kernel's LDS",
                d.d_k, d.d_v);
  C.kern = kern;
  const int rows_per_block = kern == Kern::Mfma128 ? mfma_d128_rows_per_block()
                             : kern == Kern::Valu  ? valu_rows_per_block()
                             : kern == Kern::Mla   ? mla_rows_per_block()
                                                   : decode_d128_max_rows();
  lp.nrb = std::max(1, (P.max_rows + rows_per_block - 1) / rows_per_block);
  lp.max_rows = P.max_rows;
  lp.n_groups = req->batch * d.n_kv_heads;
  lp.n_xcd = s->shape.xcds;
  if (kern == Kern::Mfma128) lp.n_groups = (int32_t)round_up(lp.n_groups, lp.n_xcd);

  int32_t splits = 1;
  const int64_t blocks = (int64_t)req->batch * d.n_kv_heads * lp.nrb;
  if (mode == Mode::Decode) {
    if (num_splits > 0) {
      splits = num_splits;
    } else {
      // about 8 work items per CU (one wave each for the decode kernel, a
      // workgroup each otherwise), never more splits than tiles
      const int64_t items = 8 * (int64_t)s->shape.cus;
      splits = (int32_t)std::max<int64_t>(1, std::min<int64_t>((items + blocks - 1) / blocks, 256));
      splits = std::min(splits, std::max(1, P.max_tiles));
    }
  } else {
    // Few row blocks per call -- short queries over long documents (the
    // regime the paper targets: a few dozen dynamic tokens after thousands
    // of cached ones), or a single small request -- leave most CUs idle and
    // let the longest request set the kernel time. Split every request's
    // key range so that its longest piece is no longer than the average work
    // per resident workgroup of the GPU (its CUs times the kernel's
    // workgroups per CU), with a minimum piece (8 tiles for the MLA kernel,
    // 1 for the vector-ALU kernel, whose tiles are slow) and at most 16
    // pieces. A piece of the d=128 matrix-core kernel only has to read more
    // keys and values than the partial results it writes and the merge
    // reads back (2 x rows x (d_v + 2) fp32), at most 8 tiles; and a d=128
    // call whose row blocks fill at most half the GPU takes as many pieces
    // as one round of workgroups holds, up to 32 (a single short request,
    // 4 links of 512 tokens and 16 questions: 15 -> 10 us), but no more: the
    // pieces of a second round cost more than they save (8 ragged requests
    // x 2 kv heads: 16 pieces 28 us, 19 pieces 41 us). Its partials then
    // stay below 256 x 256 rows x (d_v + 2) fp32 (34 MB).
    const int64_t per_cu =
        kern == Kern::Mla ? 1 : kern == Kern::Mfma128 ? mfma_d128_blocks_per_cu() : 4;
    const int64_t slots = (int64_t)s->shape.cus * per_cu;
    int min_piece = kern == Kern::Valu ? 1 : 8;
    int64_t max_splits = 16;
    if (kern == Kern::Mfma128) {
      const int64_t part = 2 * (int64_t)std::min(P.max_rows, rows_per_block) * (d.d_v + 2) * 4;
      const int64_t tile = (int64_t)kTile * (d.d_k + d.d_v) * s->esz;
      min_piece = (int)std::max<int64_t>(1, std::min<int64_t>(8, part / tile));
      if (2 * blocks <= slots) max_splits = std::min<int64_t>(32, slots / blocks);
    }
    int64_t work = 0;   // tiles summed over all non-empty workgroups
    for (const ReqEntry &R : P.reqs) {
      const int64_t rows = (int64_t)R.lq * lp.group;
      work += (int64_t)d.n_kv_heads * ((rows + rows_per_block - 1) / rows_per_block) * R.tiles;
    }
    const int64_t per_slot = std::max<int64_t>(min_piece, (work + slots - 1) / slots);
    splits = (int32_t)std::min<int64_t>(max_splits, (P.max_tiles + per_slot - 1) / per_slot);
    splits = std::max(1, std::min(splits, P.max_tiles / min_piece));
  }
  // A small generic call of a shape the lean kernel is built for (tables as
  // a kernel argument, at most kLeanTiles tiles in all) runs it.
  if (kern == Kern::Valu && !mla && lean_supported(d.dtype, d.d_k, d.d_v, lp.group) &&
      P.links.size() <= (size_t)kSmallLinks && P.reqs.size() <= (size_t)kSmallReqs &&
      P.doc_lim.empty()) {
    int64_t tiles = 0;
    for (const ReqEntry &R : P.reqs) tiles += R.tiles;
    C.lean = tiles <= kLeanTiles;
  }
  C.splits = splits;
  lp.num_splits = splits;
  if (kern == Kern::Mfma128 && splits == 1)
    balance_order_d128(s, P, lp, rows_per_block,
                       s->shape.cus / s->shape.xcds * mfma_d128_blocks_per_cu());
  const size_t rows = (size_t)P.total_q * n_q_heads;
  C.part_off = round_up(P.own_bytes, 256);
  C.part_bytes = splits > 1 ? rows * splits * (d.d_v + 2) * sizeof(float) : 0;
  return PIC_OK;
}

// Enqueues a call whose tables are already on the device (lp.links, reqs,
// order set): own-KV staging, the attention kernel, the split combine.
// timed: the attention launch may be bracketed by the measurement events
// (pic_prof_begin); the entry point that allocates nothing passes false.
pic_status launch_call(const pic_store *s, const Setup &C, LinkParams lp, void *work,
                       const Prologue &pro, const void *q, const void *k_self,
                       const void *v_self, float scale, void *out, float *lse, hipStream_t st,
                       bool timed = true) {
  const pic_store_desc &d = s->desc;
  const bool mla = d.kind == PIC_MLA;
  lp.q = q;
  lp.k_self = k_self;
  lp.v_self = v_self;
  lp.out = out;
  lp.lse = lse;
  lp.scale_log2 = scale * 1.4426950408889634f;
  if (C.splits > 1) {
    const size_t rows = (size_t)C.P.total_q * lp.n_q_heads;
    lp.part_o = (float *)((char *)work + C.part_off);
    lp.part_m = lp.part_o + rows * C.splits * d.d_v;
    lp.part_l = lp.part_m + rows * C.splits;
  }
  if (C.P.max_own_lp > 0 || pro.copy_bytes > 0) {
    hipError_t e = launch_prologue(lp, pro.links, pro.reqs, mla, s->esz, C.P.max_own_lp,
                                   C.own_args.empty() ? nullptr : C.own_args.data(), work,
                                   pro.copy_src, pro.copy_dst, pro.copy_bytes, st);
    if (e != hipSuccess) return hip_fail(e, "prep_own_kernel");
  }
  std::pair<hipEvent_t, hipEvent_t> ev{nullptr, nullptr};
  const char *name = "";
  if (timed) prof_start(st, &ev);
  hipError_t e;
  if (C.kern == Kern::Decode128)
    e = launch_link_decode_d128(lp, st, &name);
  else if (C.kern == Kern::Mla)
    e = launch_link_mla(lp, st, &name);
  else if (C.kern == Kern::Mfma128)
    e = launch_link_mfma_d128(lp, st, &name);
  else
    e = launch_link_valu(lp, d.dtype, mla, st, &name);
  prof_stop(st, &ev, name);
  if (e != hipSuccess) return hip_fail(e, name);
  if (C.splits > 1) {
    e = launch_combine(lp, d.dtype, st);
    if (e != hipSuccess) return hip_fail(e, "combine_kernel");
  }
  return PIC_OK;
}

// A generic-kernel call small enough for its tables to travel as a kernel
// argument (SmallTabs) skips the prologue: link_small_kernel reads its
// tables from its arguments and its own-KV tiles from k_self / v_self. For
// latency-bound calls the prologue was a sixth of the step (tiny_f32: 3.7
// of 23.4 us).
bool small_call(const Setup &C) {
  return C.kern == Kern::Valu && C.P.links.size() <= (size_t)kSmallLinks &&
         C.P.reqs.size() <= (size_t)kSmallReqs && C.P.doc_lim.empty();
}

// A small call's kernels: the tables go as a kernel argument and the own KV
// is read in place, so the only device memory besides the caller's tensors
// is `work` for the split partials (C.part_bytes, unused when not split).
// links: host, C.P.links.size() entries (C.P.links, or a plan's for one
// layer).
pic_status launch_small(const pic_store_desc &d, const Setup &C, const LinkEntry *links,
                        void *work, const void *q, const void *k_self, const void *v_self,
                        float scale, void *out, float *lse, hipStream_t st) {
  LinkParams lp = C.lp;
  if (C.splits > 1) {
    const size_t rows = (size_t)C.P.total_q * lp.n_q_heads;
    lp.part_o = (float *)work;
    lp.part_m = lp.part_o + rows * C.splits * d.d_v;
    lp.part_l = lp.part_m + rows * C.splits;
  }
  lp.links = nullptr;
  lp.reqs = nullptr;
  lp.order = nullptr;
  lp.doc_lim = nullptr;
  lp.q = q;
  lp.k_self = k_self;
  lp.v_self = v_self;
  lp.out = out;
  lp.lse = lse;
  lp.scale_log2 = scale * 1.4426950408889634f;
  std::pair<hipEvent_t, hipEvent_t> ev{nullptr, nullptr};
  const char *name = "";
  hipError_t e;
  if (C.lean) {
    LeanTabs t;
    memset(&t, 0, sizeof(t));
    std::copy(links, links + C.P.links.size(), t.links);
    int32_t base = 0;
    for (size_t i = 0; i < C.P.order.size(); ++i) {
      const ReqEntry &R = C.P.reqs[C.P.order[i]];
      t.reqs[i] = R;
      t.tile_base[i] = base;
      for (int32_t k = 0; k < R.nlinks; ++k) {
        const LinkEntry &L = links[R.link0 + k];
        const int32_t n = (L.len + kTile - 1) / kTile;
        for (int32_t j = 0; j < n; ++j) t.tile_link[base + L.tile0 + j] = (uint8_t)k;
      }
      base += R.tiles;
    }
    prof_start(st, &ev);
    e = launch_link_lean(lp, t, d.dtype, st, &name);
  } else {
    SmallTabs t;
    memset(&t, 0, sizeof(t));
    std::copy(links, links + C.P.links.size(), t.links);
    std::copy(C.P.reqs.begin(), C.P.reqs.end(), t.reqs);
    std::copy(C.P.order.begin(), C.P.order.end(), t.order);
    prof_start(st, &ev);
    e = launch_link_small(lp, t, d.dtype, d.kind == PIC_MLA, st, &name);
  }
  prof_stop(st, &ev, name);
  if (e != hipSuccess) return hip_fail(e, name);
  if (C.splits > 1) {
    e = launch_combine(lp, d.dtype, st);
    if (e != hipSuccess) return hip_fail(e, "combine_kernel");
  }
  return PIC_OK;
}

pic_status small_link_call(pic_store *s, const Setup &C, const void *q, const void *k_self,
                           const void *v_self, float scale, void *out, float *lse,
                           hipStream_t st) {
  Stage *stage = nullptr;
  pic_status rc = stage_acquire(s, 0, &stage);
  if (rc != PIC_OK) return rc;
  if (C.splits > 1) {
    rc = ensure_work(stage, C.part_bytes);
    if (rc != PIC_OK) return rc;
  }
  rc = launch_small(s->desc, C, C.P.links.data(), stage->work, q, k_self, v_self, scale, out,
                    lse, st);
  if (rc != PIC_OK) return rc;
  HIP_TRY(hipEventRecord(stage->done, st), "hipEventRecord(stage)");
  stage->pending = true;
  return PIC_OK;
}

pic_status link_call(pic_store *s, const pic_link_req *req, int32_t n_q_heads, const void *q,
                     const void *k_self, const void *v_self, float scale, int32_t num_splits,
                     void *out, float *lse, void *stream, Mode mode) {
  if (!req) return fail(PIC_ERR_INVALID, "req is NULL");
  Setup C;
  pic_status rc = setup_call(s, req, n_q_heads, scale, req->layer, num_splits, mode, C);
  if (rc != PIC_OK) return rc;
  if (req->batch == 0) return PIC_OK;
  rc = check_tensors(s, C.P, q, k_self, v_self, out);
  if (rc != PIC_OK) return rc;
  if (C.P.total_q == 0) return PIC_OK;
  const hipStream_t st = (hipStream_t)stream;
  // the workspace is allocated on the store's device
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  if (small_call(C)) return small_link_call(s, C, q, k_self, v_self, scale, out, lse, st);
  Stage *stage = nullptr;
  TableLayout tl;
  LinkParams lp = C.lp;
  rc = upload(s, C.P, C.work_bytes(), &stage, lp, tl);
  if (rc != PIC_OK) return rc;
  Prologue pro;
  const char *hd = (const char *)stage->host_dev;
  pro.links = (const LinkEntry *)hd;
  pro.reqs = (const ReqEntry *)(hd + tl.off_r);
  pro.copy_src = hd;
  pro.copy_dst = stage->dev;
  pro.copy_bytes = (int64_t)tl.bytes;
  rc = launch_call(s, C, lp, stage->work, pro, q, k_self, v_self, scale, out, lse, st);
  if (rc != PIC_OK) return rc;
  HIP_TRY(hipEventRecord(stage->done, st), "hipEventRecord(stage)");
  stage->pending = true;
  return PIC_OK;
}

}  // namespace

// A request batch resolved once for repeated calls: the link tables of every
// layer and the call's workspace live on the device for the plan's lifetime.
struct pic_link_plan {
  pic_store *store = nullptr;
  Setup C;
  int32_t batch = 0;
  void *dev = nullptr;           // [layer tables][workspace]
  size_t table_bytes = 0;        // one layer's tables, 256-byte aligned
  size_t off_r = 0, off_o = 0;   // request / order tables within a layer's tables
  size_t off_d = 0;              // per-query limits (if any) within a layer's tables
  void *work = nullptr;          // inside dev
  // small calls (see small_call): every layer's link table on the host,
  // [layer][link], run by the small-call kernels as pic_link_attn /
  // pic_link_decode run them (tables as a kernel argument)
  bool small = false;
  std::vector<LinkEntry> small_links;
};

extern "C" {

pic_status pic_store_create(const pic_store_desc *desc, pic_store **out) {
  if (!desc || !out) return fail(PIC_ERR_INVALID, "desc/out is NULL");
  *out = nullptr;
  const pic_store_desc &d = *desc;
  if (d.kind != PIC_GQA && d.kind != PIC_MLA) return fail(PIC_ERR_INVALID, "unknown kind %d", d.kind);
  if (d.dtype != PIC_F32 && d.dtype != PIC_BF16) return fail(PIC_ERR_INVALID, "unknown dtype %d", d.dtype);
  if (d.n_layers < 0 || d.n_layers > 256) return fail(PIC_ERR_INVALID, "n_layers must be 0..256");
  if (d.n_kv_heads <= 0 || d.d_k <= 0 || d.d_v <= 0 || d.capacity_tokens <= 0)
    return fail(PIC_ERR_INVALID, "n_kv_heads, d_k, d_v and capacity_tokens must be positive");
  if (d.kind == PIC_MLA && (d.n_kv_heads != 1 || d.d_v > d.d_k))
    return fail(PIC_ERR_INVALID, "MLA needs n_kv_heads == 1 and d_v <= d_k");
  if (d.d_k % 8 || d.d_v % 8) return fail(PIC_ERR_UNSUPPORTED, "d_k and d_v must be multiples of 8");
  if (d.d_k > 1024 || d.d_v > 1024 || d.n_kv_heads > 256)
    return fail(PIC_ERR_UNSUPPORTED, "head count or width too large");
  pic_store *s = new (std::nothrow) pic_store();
  if (!s) return fail(PIC_ERR_OOM, "host allocation failed");
  s->desc = d;
  s->esz = d.dtype == PIC_F32 ? 4 : 2;
  s->capacity = round_up(d.capacity_tokens, kTile);
  s->k_tok_elems = (int64_t)d.n_kv_heads * d.d_k;
  s->v_tok_elems = d.kind == PIC_GQA ? (int64_t)d.n_kv_heads * d.d_v : 0;
  s->n_layers = d.n_layers > 1 ? d.n_layers : 1;
  s->layer_bytes = s->capacity * (s->k_tok_elems + s->v_tok_elems) * s->esz;
  s->free_runs.emplace(0, s->capacity / kTile);
  hipError_t e = hipGetDevice(&s->device);
  if (e == hipSuccess) s->shape = device_shape();
  if (e == hipSuccess) e = hipMalloc((void **)&s->pool, (size_t)s->layer_bytes * s->n_layers);
  if (e != hipSuccess) {
    delete s;
    return hip_fail(e, "hipMalloc(pool)");
  }
  try {
    s->page_refs.assign((size_t)(s->capacity / kTile), 0);
  } catch (...) {
    (void)hipFree(s->pool);
    delete s;
    return fail(PIC_ERR_OOM, "host allocation failed");
  }
  *out = s;
  return PIC_OK;
}

pic_status pic_store_destroy(pic_store *s) {
  if (!s) return PIC_OK;
  if (s->live_plans > 0)
    return fail(PIC_ERR_INVALID, "%lld link plans of this store are still alive",
                (long long)s->live_plans);
  DeviceGuard dg(s->device);
  (void)hipDeviceSynchronize();
  for (Stage &st : s->ring) {
    if (st.host) (void)hipHostFree(st.host);
    if (st.dev) (void)hipFree(st.dev);
    if (st.work) (void)hipFree(st.work);
    if (st.done) (void)hipEventDestroy(st.done);
  }
  for (auto &pr : s->pending) (void)hipEventDestroy(pr.first);
  if (s->pool) {
    if (s->imported)
      (void)hipIpcCloseMemHandle(s->pool);
    else
      (void)hipFree(s->pool);
  }
  delete s;
  return PIC_OK;
}

pic_status pic_store_put(pic_store *s, uint64_t chunk_id, int64_t n_tokens, const void *k,
                         const void *v, void *stream) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (s->imported) return fail(PIC_ERR_INVALID, "the store was imported from another process and is read-only");
  if (n_tokens <= 0 || n_tokens > INT32_MAX / 4) return fail(PIC_ERR_INVALID, "n_tokens out of range");
  if (!k) return fail(PIC_ERR_INVALID, "k is NULL");
  const bool gqa = s->desc.kind == PIC_GQA;
  if (gqa && !v) return fail(PIC_ERR_INVALID, "v is NULL");
  if (!gqa && v) return fail(PIC_ERR_INVALID, "v must be NULL for MLA");
  if (s->map.count(chunk_id)) return fail(PIC_ERR_EXISTS, "chunk id 0x%llx already stored",
                                          (unsigned long long)chunk_id);
  const int64_t pages = round_up(n_tokens, kTile) / kTile;
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  for (const void *ptr : {k, v}) {
    if (!ptr) continue;
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, ptr) != hipSuccess ||
        (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged)) {
      (void)hipGetLastError();
      return fail(PIC_ERR_INVALID, "k and v must be device memory");
    }
  }
  std::vector<Run> runs;
  pic_status rc = take_pages(s, pages, runs);
  if (rc != PIC_OK) return rc;
  int32_t tok = 0;
  for (Run &r : runs) {
    r.tok0 = tok;
    r.ntok = (int32_t)std::min<int64_t>((int64_t)r.pages * kTile, n_tokens - tok);
    tok += r.ntok;
  }
  const hipStream_t st = (hipStream_t)stream;
  const pic_store_desc &d = s->desc;
  // layer l of the caller's buffers -> layer l of each run
  const int64_t k_src_layer = n_tokens * s->k_tok_elems * s->esz;
  const int64_t v_src_layer = n_tokens * s->v_tok_elems * s->esz;
  hipError_t e = hipSuccess;
  for (int32_t l = 0; l < s->n_layers && e == hipSuccess; ++l) {
    for (const Run &r : runs) {
      const LinkEntry E = run_entry(s, r, l);
      const char *ksrc = (const char *)k + l * k_src_layer + (int64_t)r.tok0 * s->k_tok_elems * s->esz;
      e = launch_put_rows(ksrc, (void *)E.k, r.ntok, E.lp, d.n_kv_heads, d.d_k, s->esz, st);
      if (e != hipSuccess) break;
      if (gqa) {
        const char *vsrc =
            (const char *)v + l * v_src_layer + (int64_t)r.tok0 * s->v_tok_elems * s->esz;
        e = launch_put_transposed(vsrc, (void *)E.v, r.ntok, E.lp, d.n_kv_heads, d.d_v, s->esz, st);
        if (e != hipSuccess) break;
      }
    }
  }
  if (e != hipSuccess) {
    for (const Run &r : runs) free_run(s, r.page0, r.pages);
    return hip_fail(e, "put kernels");
  }
  Slot sl;
  sl.len = n_tokens;
  for (const Run &r : runs) s->block_refs[r.page0] = 1;
  ref_pages(s, runs, 1);
  sl.runs = std::move(runs);
  s->used += pages * kTile;
  s->map.emplace(chunk_id, std::move(sl));
  return PIC_OK;
}

pic_status pic_store_derive(pic_store *s, uint64_t new_id, uint64_t base_id, int32_t n_rows,
                            const int32_t *rows, void *stream) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (s->imported) return fail(PIC_ERR_INVALID, "the store was imported from another process and is read-only");
  auto bit = s->map.find(base_id);
  if (bit == s->map.end()) return fail(PIC_ERR_NOT_FOUND, "base chunk id 0x%llx not in the store",
                                       (unsigned long long)base_id);
  if (s->map.count(new_id)) return fail(PIC_ERR_EXISTS, "chunk id 0x%llx already stored",
                                        (unsigned long long)new_id);
  const int64_t len = bit->second.len;
  if (!check_rows(rows, n_rows, len))
    return fail(PIC_ERR_INVALID, "rows must be strictly increasing and below the chunk's %lld tokens",
                (long long)len);
  const int64_t npages = round_up(len, kTile) / kTile;
  std::vector<char> own(npages, 0);
  int64_t n_own = 0;
  for (int32_t i = 0; i < n_rows; ++i) {
    char &o = own[rows[i] / kTile];
    n_own += !o;
    o = 1;
  }
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  std::vector<Run> fresh;
  pic_status rc = take_pages(s, n_own, fresh);
  if (rc != PIC_OK) return rc;
  const Slot &B = s->map.at(base_id);   // take_pages does not touch the map
  // One view per chunk page, merged where consecutive pages are consecutive
  // pages of one block; private pages take the fresh blocks' pages in order.
  std::vector<Run> views;
  std::vector<std::pair<Run, Run>> copies;     // (source page view, destination page view)
  size_t fb = 0;
  int32_t fq = 0;
  for (int64_t p = 0; p < npages; ++p) {
    const int32_t t0 = (int32_t)(p * kTile);
    const int32_t nt = (int32_t)std::min<int64_t>(kTile, len - t0);
    const Run &src = view_of(B, t0);
    Run pv{src.page0, src.pages, t0, nt, src.skip + (t0 - src.tok0) / kTile};
    if (own[p]) {
      Run dst{fresh[fb].page0, fresh[fb].pages, t0, nt, fq};
      copies.emplace_back(pv, dst);
      pv = dst;
      if (++fq == fresh[fb].pages) {
        ++fb;
        fq = 0;
      }
    }
    if (!views.empty()) {
      Run &last = views.back();
      if (last.page0 == pv.page0 && last.skip + last.ntok / kTile == pv.skip && last.ntok % kTile == 0) {
        last.ntok += nt;
        continue;
      }
    }
    views.push_back(pv);
  }
  // copy the private pages' base content, every layer (K rows of each head,
  // V^T columns of each head and dim)
  const hipStream_t st = (hipStream_t)stream;
  const pic_store_desc &d = s->desc;
  hipError_t e = hipSuccess;
  for (int32_t l = 0; l < s->n_layers && e == hipSuccess; ++l)
    for (const auto &c : copies) {
      const LinkEntry S = run_entry(s, c.first, l), D = run_entry(s, c.second, l);
      const size_t kw = (size_t)kTile * d.d_k * s->esz;
      e = hipMemcpy2DAsync((void *)D.k, (size_t)D.lp * d.d_k * s->esz, S.k,
                           (size_t)S.lp * d.d_k * s->esz, kw, (size_t)d.n_kv_heads,
                           hipMemcpyDeviceToDevice, st);
      if (e != hipSuccess) break;
      if (d.kind == PIC_GQA) {   // a page is two whole V^T panels per head
        e = hipMemcpy2DAsync((void *)D.v, (size_t)D.lp * d.d_v * s->esz, S.v,
                             (size_t)S.lp * d.d_v * s->esz, (size_t)kTile * d.d_v * s->esz,
                             (size_t)d.n_kv_heads, hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) break;
      }
    }
  if (e != hipSuccess) {
    for (const Run &r : fresh) free_run(s, r.page0, r.pages);
    return hip_fail(e, "derive page copies");
  }
  for (const Run &r : fresh) s->block_refs[r.page0] = 0;
  std::vector<int64_t> blocks;
  for (const Run &v : views) blocks.push_back(v.page0);
  std::sort(blocks.begin(), blocks.end());
  blocks.erase(std::unique(blocks.begin(), blocks.end()), blocks.end());
  for (int64_t b : blocks) ++s->block_refs.at(b);
  ref_pages(s, views, 1);
  s->used += n_own * kTile;
  Slot sl;
  sl.len = len;
  sl.runs = std::move(views);
  sl.derived = true;
  s->map.emplace(new_id, std::move(sl));
  return PIC_OK;
}

pic_status pic_store_write_rows(pic_store *s, uint64_t chunk_id, int32_t layer, int32_t n_rows,
                                const int32_t *rows, const void *k, const void *v, void *stream) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (s->imported) return fail(PIC_ERR_INVALID, "the store was imported from another process and is read-only");
  auto it = s->map.find(chunk_id);
  if (it == s->map.end()) return fail(PIC_ERR_NOT_FOUND, "chunk id 0x%llx not in the store",
                                      (unsigned long long)chunk_id);
  const Slot &sl = it->second;
  if (!sl.derived)
    return fail(PIC_ERR_INVALID, "chunk id 0x%llx was not made by pic_store_derive",
                (unsigned long long)chunk_id);
  if (layer < 0 || layer >= s->n_layers)
    return fail(PIC_ERR_INVALID, "layer %d outside the store's %d layers", layer, s->n_layers);
  if (!check_rows(rows, n_rows, sl.len))
    return fail(PIC_ERR_INVALID, "rows must be strictly increasing and below the chunk's %lld tokens",
                (long long)sl.len);
  if (n_rows == 0) return PIC_OK;
  const bool gqa = s->desc.kind == PIC_GQA;
  if (!k || (gqa && !v)) return fail(PIC_ERR_INVALID, "k/v is NULL");
  if (!gqa && v) return fail(PIC_ERR_INVALID, "v must be NULL for MLA");
  std::vector<RowDst> dst(n_rows);
  for (int32_t i = 0; i < n_rows; ++i) {
    const Run &r = view_of(sl, rows[i]);
    if (s->page_refs[r.page0 + r.skip + (rows[i] - r.tok0) / kTile] != 1)
      return fail(PIC_ERR_INVALID, "row %d of chunk 0x%llx is on a page shared with another chunk",
                  rows[i], (unsigned long long)chunk_id);
    const LinkEntry E = run_entry(s, r, layer);
    const int64_t t = rows[i] - r.tok0;
    dst[i].k = (char *)E.k + t * s->desc.d_k * s->esz;
    dst[i].v = gqa ? (char *)E.v + vt_offset(0, 0, t, E.lp, s->desc.d_v) * s->esz : nullptr;
    dst[i].lp = E.lp;
  }
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  const hipStream_t st = (hipStream_t)stream;
  const size_t bytes = sizeof(RowDst) * (size_t)n_rows;
  Stage *stage = nullptr;
  pic_status rc = stage_acquire(s, bytes, &stage);
  if (rc != PIC_OK) return rc;
  memcpy(stage->host, dst.data(), bytes);
  HIP_TRY(launch_table_copy(stage->host_dev, stage->dev, (int64_t)round_up(bytes, 16), st),
          "table_copy_kernel");
  const pic_store_desc &d = s->desc;
  HIP_TRY(launch_write_rows((const RowDst *)stage->dev, n_rows, k, v, d.n_kv_heads, d.d_k, d.d_v,
                            !gqa, s->esz, st),
          "write_rows_kernel");
  HIP_TRY(hipEventRecord(stage->done, st), "hipEventRecord(stage)");
  stage->pending = true;
  return PIC_OK;
}

pic_status pic_store_remove(pic_store *s, uint64_t chunk_id, void *stream) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (s->imported) return fail(PIC_ERR_INVALID, "the store was imported from another process and is read-only");
  auto it = s->map.find(chunk_id);
  if (it == s->map.end()) return fail(PIC_ERR_NOT_FOUND, "chunk id 0x%llx not in the store",
                                      (unsigned long long)chunk_id);
  if (it->second.plan_refs > 0)
    return fail(PIC_ERR_INVALID, "chunk id 0x%llx is linked by %lld live link plans",
                (unsigned long long)chunk_id, (long long)it->second.plan_refs);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  // the pages are reused only after the work enqueued so far on `stream`
  // (the calls that may read them) has completed
  hipEvent_t ev = nullptr;
  HIP_TRY(hipEventCreateWithFlags(&ev, hipEventDisableTiming), "hipEventCreate(remove)");
  hipError_t e = hipEventRecord(ev, (hipStream_t)stream);
  if (e != hipSuccess) {
    (void)hipEventDestroy(ev);
    return hip_fail(e, "hipEventRecord(remove)");
  }
  // blocks no other chunk views are freed once the event has completed
  ref_pages(s, it->second.runs, -1);
  std::vector<Run> freed;
  std::vector<int64_t> blocks;
  for (const Run &r : it->second.runs) blocks.push_back(r.page0);
  std::sort(blocks.begin(), blocks.end());
  blocks.erase(std::unique(blocks.begin(), blocks.end()), blocks.end());
  for (int64_t b : blocks) {
    auto ref = s->block_refs.find(b);
    if (--ref->second > 0) continue;
    const Run &r = *std::find_if(it->second.runs.begin(), it->second.runs.end(),
                                 [b](const Run &x) { return x.page0 == b; });
    freed.push_back(Run{r.page0, r.pages, 0, 0});
    s->block_refs.erase(ref);
  }
  if (freed.empty())
    (void)hipEventDestroy(ev);
  else
    s->pending.emplace_back(ev, std::move(freed));
  s->map.erase(it);
  return PIC_OK;
}

namespace {

// Layout of an exported store: header, then per chunk its record and runs.
constexpr uint64_t kExportMagic = 0x31524f5453434950ull;   // "PICSTOR1"
struct ExportHeader {
  uint64_t magic;
  uint64_t bytes;                // whole blob
  pic_store_desc desc;
  int64_t capacity, layer_bytes, k_tok_elems, v_tok_elems, used, n_chunks;
  int32_t n_layers, esz;
  hipIpcMemHandle_t handle;      // the pool
};
struct ExportChunk {
  uint64_t id;
  int64_t len;
  int32_t n_runs, derived;
};
struct ExportRun {
  int64_t page0;
  int32_t pages, tok0, ntok, skip;
};

// Pools from 2 GiB up are not exported: opening such a mapping in another
// process has not returned on the target machines.
constexpr int64_t kMaxExportBytes = (int64_t(1) << 31) - 1;

size_t export_size(const pic_store *s) {
  size_t n = sizeof(ExportHeader);
  for (const auto &kv : s->map) n += sizeof(ExportChunk) + kv.second.runs.size() * sizeof(ExportRun);
  return n;
}

}  // namespace

pic_status pic_store_export(pic_store *s, void *buf, size_t buf_bytes, size_t *bytes_out) {
  if (!s || !bytes_out) return fail(PIC_ERR_INVALID, "store/bytes_out is NULL");
  if (s->imported) return fail(PIC_ERR_INVALID, "an imported store cannot be exported again");
  const int64_t pool_bytes = s->layer_bytes * s->n_layers;
  if (pool_bytes > kMaxExportBytes)
    return fail(PIC_ERR_UNSUPPORTED, "pool of %lld bytes: only pools below 2 GiB are exported",
                (long long)pool_bytes);
  const size_t need = export_size(s);
  *bytes_out = need;
  if (!buf) return PIC_OK;
  if (buf_bytes < need) return fail(PIC_ERR_INVALID, "buffer of %zu bytes, %zu needed", buf_bytes, need);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  // every put and copy enqueued so far lands before another process reads
  HIP_TRY(hipDeviceSynchronize(), "hipDeviceSynchronize(export)");
  ExportHeader h{};
  h.magic = kExportMagic;
  h.bytes = need;
  h.desc = s->desc;
  h.capacity = s->capacity;
  h.layer_bytes = s->layer_bytes;
  h.k_tok_elems = s->k_tok_elems;
  h.v_tok_elems = s->v_tok_elems;
  h.used = s->used;
  h.n_chunks = (int64_t)s->map.size();
  h.n_layers = s->n_layers;
  h.esz = s->esz;
  HIP_TRY(hipIpcGetMemHandle(&h.handle, s->pool), "hipIpcGetMemHandle(pool)");
  char *o = (char *)buf;
  memcpy(o, &h, sizeof h);
  o += sizeof h;
  for (const auto &kv : s->map) {
    const ExportChunk ch{kv.first, kv.second.len, (int32_t)kv.second.runs.size(),
                         kv.second.derived ? 1 : 0};
    memcpy(o, &ch, sizeof ch);
    o += sizeof ch;
    for (const Run &r : kv.second.runs) {
      const ExportRun er{r.page0, r.pages, r.tok0, r.ntok, r.skip};
      memcpy(o, &er, sizeof er);
      o += sizeof er;
    }
  }
  return PIC_OK;
}

pic_status pic_store_import(const void *buf, size_t buf_bytes, pic_store **out) {
  if (!buf || !out) return fail(PIC_ERR_INVALID, "buf/out is NULL");
  *out = nullptr;
  ExportHeader h;
  if (buf_bytes < sizeof h) return fail(PIC_ERR_INVALID, "blob too short");
  memcpy(&h, buf, sizeof h);
  if (h.magic != kExportMagic) return fail(PIC_ERR_INVALID, "not an exported store");
  if (h.bytes > buf_bytes || h.n_chunks < 0 || h.n_layers < 1 || h.n_layers > 256 ||
      (h.esz != 2 && h.esz != 4) || h.capacity <= 0 || h.capacity % kTile ||
      h.layer_bytes != h.capacity * (h.k_tok_elems + h.v_tok_elems) * h.esz ||
      h.layer_bytes * h.n_layers > kMaxExportBytes)
    return fail(PIC_ERR_INVALID, "inconsistent exported store header");
  const int64_t pages = h.capacity / kTile;
  pic_store *s = new (std::nothrow) pic_store();
  if (!s) return fail(PIC_ERR_OOM, "host allocation failed");
  s->desc = h.desc;
  s->esz = h.esz;
  s->capacity = h.capacity;
  s->used = h.used;
  s->k_tok_elems = h.k_tok_elems;
  s->v_tok_elems = h.v_tok_elems;
  s->n_layers = h.n_layers;
  s->layer_bytes = h.layer_bytes;
  const char *in = (const char *)buf + sizeof h, *end = (const char *)buf + h.bytes;
  for (int64_t c = 0; c < h.n_chunks; ++c) {
    ExportChunk ch;
    if (in + sizeof ch > end) break;
    memcpy(&ch, in, sizeof ch);
    in += sizeof ch;
    if (ch.n_runs < 1 || ch.len < 1 || in + (size_t)ch.n_runs * sizeof(ExportRun) > end) {
      delete s;
      return fail(PIC_ERR_INVALID, "corrupt chunk record in the exported store");
    }
    Slot sl;
    sl.len = ch.len;
    sl.derived = ch.derived != 0;
    int64_t covered = 0;
    for (int32_t i = 0; i < ch.n_runs; ++i) {
      ExportRun er;
      memcpy(&er, in, sizeof er);
      in += sizeof er;
      // every view lies inside the pool and the views cover the chunk in order
      if (er.page0 < 0 || er.pages < 1 || er.page0 + er.pages > pages || er.skip < 0 ||
          er.ntok < 1 || er.tok0 != covered ||
          (int64_t)er.skip * kTile + er.ntok > (int64_t)er.pages * kTile) {
        delete s;
        return fail(PIC_ERR_INVALID, "corrupt run in the exported store");
      }
      covered += er.ntok;
      sl.runs.push_back(Run{er.page0, er.pages, er.tok0, er.ntok, er.skip});
    }
    if (covered != ch.len || !s->map.emplace(ch.id, std::move(sl)).second) {
      delete s;
      return fail(PIC_ERR_INVALID, "corrupt chunk record in the exported store");
    }
  }
  if ((int64_t)s->map.size() != h.n_chunks) {
    delete s;
    return fail(PIC_ERR_INVALID, "truncated exported store");
  }
  hipError_t e = hipGetDevice(&s->device);
  if (e == hipSuccess) {
    s->shape = device_shape();
    e = hipIpcOpenMemHandle((void **)&s->pool, h.handle, hipIpcMemLazyEnablePeerAccess);
  }
  if (e != hipSuccess) {
    delete s;
    return hip_fail(e, "hipIpcOpenMemHandle(pool)");
  }
  s->imported = true;
  *out = s;
  return PIC_OK;
}

pic_status pic_store_lookup(const pic_store *s, uint64_t chunk_id, int64_t *n_tokens_out) {
  if (!s || !n_tokens_out) return fail(PIC_ERR_INVALID, "store/n_tokens_out is NULL");
  auto it = s->map.find(chunk_id);
  if (it == s->map.end()) return fail(PIC_ERR_NOT_FOUND, "chunk id 0x%llx not in the store",
                                      (unsigned long long)chunk_id);
  *n_tokens_out = it->second.len;
  return PIC_OK;
}

pic_status pic_store_usage(const pic_store *s, int64_t *used, int64_t *cap, int64_t *n) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (used) *used = s->used;
  if (cap) *cap = s->capacity;
  if (n) *n = (int64_t)s->map.size();
  return PIC_OK;
}

pic_status pic_link_attn(pic_store *s, const pic_link_req *req, int32_t n_q_heads, const void *q,
                         const void *k_self, const void *v_self, float softmax_scale, void *out,
                         float *lse, void *stream) {
  return link_call(s, req, n_q_heads, q, k_self, v_self, softmax_scale, 0, out, lse, stream,
                   Mode::Prefill);
}

pic_status pic_link_decode(pic_store *s, const pic_link_req *req, int32_t n_q_heads,
                           const void *q, const void *k_self, const void *v_self,
                           float softmax_scale, int32_t num_splits, void *out, float *lse,
                           void *stream) {
  return link_call(s, req, n_q_heads, q, k_self, v_self, softmax_scale, num_splits, out, lse,
                   stream, Mode::Decode);
}

pic_status pic_link_decode_noalloc(pic_store *s, const pic_link_req *req, int32_t n_q_heads,
                                   const void *q, const void *k_self, const void *v_self,
                                   float softmax_scale, int32_t num_splits, void *out, float *lse,
                                   void *stream) {
  if (!req) return fail(PIC_ERR_INVALID, "req is NULL");
  Setup C;
  pic_status rc = setup_call(s, req, n_q_heads, softmax_scale, req->layer, num_splits,
                             Mode::Decode, C);
  if (rc != PIC_OK) return rc;
  if (req->batch == 0) return PIC_OK;
  rc = check_tensors(s, C.P, q, k_self, v_self, out);
  if (rc != PIC_OK) return rc;
  if (C.P.total_q == 0) return PIC_OK;
  // A small call runs the kernels pic_link_decode runs for it (tables as a
  // kernel argument, own KV read in place): the scratch holds only its
  // split partials.
  if (small_call(C)) {
    if (C.part_bytes > kStaticScratchBytes)
      return fail(PIC_ERR_INVALID,
                  "the call needs %zu bytes of scratch (split partials); the static scratch "
                  "holds %zu", C.part_bytes, kStaticScratchBytes);
    DeviceGuard dg(s->device);
    if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
    void *base = nullptr;
    HIP_TRY(static_scratch(&base), "hipGetSymbolAddress(scratch)");
    return launch_small(s->desc, C, C.P.links.data(), base, q, k_self, v_self, softmax_scale,
                        out, lse, (hipStream_t)stream);
  }
  // scratch layout: [link table][request table][order][per-query limits][workspace]
  Plan &P = C.P;
  const size_t nl = P.links.size(), nr = P.reqs.size();
  const size_t off_r = round_up(sizeof(LinkEntry) * nl, 256);
  const size_t off_o = off_r + round_up(sizeof(ReqEntry) * nr, 256);
  const size_t off_d = off_o + round_up(sizeof(int32_t) * nr, 256);
  const size_t tables = off_d + round_up(sizeof(int32_t) * P.doc_lim.size(), 256);
  const size_t need = tables + C.work_bytes();
  if (need > kStaticScratchBytes)
    return fail(PIC_ERR_INVALID,
                "the call needs %zu bytes of scratch (tables, own KV, split partials); the static "
                "scratch holds %zu", need, kStaticScratchBytes);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  void *base = nullptr;
  HIP_TRY(static_scratch(&base), "hipGetSymbolAddress(scratch)");
  char *dev = (char *)base;
  place_own(s, P, dev + tables, P.links.data());
  std::vector<char> host(tables, 0);
  if (nl) memcpy(host.data(), P.links.data(), sizeof(LinkEntry) * nl);
  memcpy(host.data() + off_r, P.reqs.data(), sizeof(ReqEntry) * nr);
  memcpy(host.data() + off_o, P.order.data(), sizeof(int32_t) * nr);
  if (!P.doc_lim.empty())
    memcpy(host.data() + off_d, P.doc_lim.data(), sizeof(int32_t) * P.doc_lim.size());
  const hipStream_t st = (hipStream_t)stream;
  // pageable source: the runtime copies it before returning (no staging
  // buffer of ours, no allocation)
  HIP_TRY(hipMemcpyAsync(dev, host.data(), tables, hipMemcpyHostToDevice, st),
          "hipMemcpyAsync(tables to scratch)");
  LinkParams lp = C.lp;
  lp.links = (const LinkEntry *)dev;
  lp.reqs = (const ReqEntry *)(dev + off_r);
  lp.order = (const int32_t *)(dev + off_o);
  lp.doc_lim = P.doc_lim.empty() ? nullptr : (const int32_t *)(dev + off_d);
  Prologue pro;
  pro.links = lp.links;
  pro.reqs = lp.reqs;
  return launch_call(s, C, lp, dev + tables, pro, q, k_self, v_self, softmax_scale, out, lse, st,
                     false);
}

pic_status pic_link_plan_create(pic_store *s, const pic_link_req *req, int32_t n_q_heads,
                                int32_t mode, int32_t num_splits, pic_link_plan **out) {
  if (!out) return fail(PIC_ERR_INVALID, "out is NULL");
  *out = nullptr;
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (!req) return fail(PIC_ERR_INVALID, "req is NULL");
  if (req->layer != 0) return fail(PIC_ERR_INVALID, "req->layer must be 0 (each run names its layer)");
  if (mode != PIC_PREFILL && mode != PIC_DECODE) return fail(PIC_ERR_INVALID, "unknown mode %d", mode);
  if (mode == PIC_PREFILL && num_splits != 0)
    return fail(PIC_ERR_INVALID, "num_splits must be 0 for prefill plans");
  pic_link_plan *pl = new (std::nothrow) pic_link_plan();
  if (!pl) return fail(PIC_ERR_OOM, "host allocation failed");
  // the scale only has to pass validation here; each run passes its own
  pic_status rc = setup_call(s, req, n_q_heads, 1.0f, 0, num_splits,
                             mode == PIC_DECODE ? Mode::Decode : Mode::Prefill, pl->C);
  if (rc != PIC_OK) {
    delete pl;
    return rc;
  }
  pl->store = s;
  pl->batch = req->batch;
  const Plan &P = pl->C.P;
  const size_t nl = P.links.size(), nr = P.reqs.size();
  pl->off_r = round_up(sizeof(LinkEntry) * nl, 256);
  pl->off_o = pl->off_r + round_up(sizeof(ReqEntry) * nr, 256);
  pl->off_d = pl->off_o + round_up(sizeof(int32_t) * nr, 256);
  pl->table_bytes = round_up(pl->off_d + sizeof(int32_t) * P.doc_lim.size(), 256);
  // A small call keeps its tables on the host (one per layer) and needs
  // device memory for its split partials only.
  pl->small = small_call(pl->C);
  if (pl->small) {
    pl->small_links.resize((size_t)s->n_layers * nl);
    std::vector<bool> own_link(nl, false);
    for (auto &o : P.own) own_link[o.first] = true;
    for (int32_t l = 0; l < s->n_layers; ++l)
      for (size_t i = 0; i < nl; ++i) {
        LinkEntry E = P.links[i];
        if (!own_link[i]) {
          E.k = (const char *)E.k + (int64_t)l * s->layer_bytes;
          E.v = (const char *)E.v + (int64_t)l * s->layer_bytes;
        }
        pl->small_links[(size_t)l * nl + i] = E;
      }
  }
  const size_t tables = pl->small ? 0 : pl->table_bytes * s->n_layers;
  const size_t bytes = pl->small ? pl->C.part_bytes : tables + pl->C.work_bytes();
  if (bytes > 0) {
    DeviceGuard dg(s->device);
    if (!dg.ok) {
      delete pl;
      return fail(PIC_ERR_HIP, "cannot select the store's device");
    }
    hipError_t e = hipMalloc(&pl->dev, bytes);
    if (e != hipSuccess) {
      delete pl;
      return hip_fail(e, "hipMalloc(plan)");
    }
    pl->work = (char *)pl->dev + tables;
  }
  if (bytes > 0 && !pl->small) {
    DeviceGuard dg(s->device);
    if (!dg.ok) {
      (void)hipFree(pl->dev);
      delete pl;
      return fail(PIC_ERR_HIP, "cannot select the store's device");
    }
    // Every layer's tables differ only in the chunk links' addresses: layer
    // l of a slot sits l pool layers further on; own-KV links point at the
    // plan's workspace in every layer.
    std::vector<char> host(tables, 0);
    std::vector<LinkEntry> links(P.links);
    place_own(s, P, pl->work, links.data());
    std::vector<bool> own(nl, false);
    for (auto &o : P.own) own[o.first] = true;
    for (int32_t l = 0; l < s->n_layers; ++l) {
      char *h = host.data() + (size_t)l * pl->table_bytes;
      LinkEntry *L = (LinkEntry *)h;
      for (size_t i = 0; i < nl; ++i) {
        L[i] = links[i];
        if (!own[i]) {
          L[i].k = (const char *)links[i].k + (int64_t)l * s->layer_bytes;
          L[i].v = (const char *)links[i].v + (int64_t)l * s->layer_bytes;
        }
      }
      if (nr) memcpy(h + pl->off_r, P.reqs.data(), sizeof(ReqEntry) * nr);
      if (nr) memcpy(h + pl->off_o, P.order.data(), sizeof(int32_t) * nr);
      if (!P.doc_lim.empty())
        memcpy(h + pl->off_d, P.doc_lim.data(), sizeof(int32_t) * P.doc_lim.size());
    }
    hipError_t e = hipMemcpy(pl->dev, host.data(), tables, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      (void)hipFree(pl->dev);
      delete pl;
      return hip_fail(e, "hipMemcpy(plan tables)");
    }
  }
  for (uint64_t id : P.ids) ++s->map.at(id).plan_refs;
  ++s->live_plans;
  *out = pl;
  return PIC_OK;
}

pic_status pic_link_plan_run(pic_link_plan *pl, int32_t layer, const void *q, const void *k_self,
                             const void *v_self, float softmax_scale, void *out, float *lse,
                             void *stream) {
  if (!pl) return fail(PIC_ERR_INVALID, "plan is NULL");
  pic_store *s = pl->store;
  if (layer < 0 || layer >= s->n_layers)
    return fail(PIC_ERR_INVALID, "layer %d outside the store's %d layers", layer, s->n_layers);
  if (!std::isfinite(softmax_scale) || !(softmax_scale > 0.f))
    return fail(PIC_ERR_INVALID, "softmax_scale must be positive and finite");
  if (pl->batch == 0) return PIC_OK;
  pic_status rc = check_tensors(s, pl->C.P, q, k_self, v_self, out);
  if (rc != PIC_OK) return rc;
  if (pl->C.P.total_q == 0) return PIC_OK;
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  if (pl->small)
    return launch_small(s->desc, pl->C,
                        pl->small_links.data() + (size_t)layer * pl->C.P.links.size(),
                        pl->work, q, k_self, v_self, softmax_scale, out, lse,
                        (hipStream_t)stream);
  LinkParams lp = pl->C.lp;
  const char *t = (const char *)pl->dev + (size_t)layer * pl->table_bytes;
  lp.links = (const LinkEntry *)t;
  lp.reqs = (const ReqEntry *)(t + pl->off_r);
  lp.order = (const int32_t *)(t + pl->off_o);
  lp.doc_lim = pl->C.P.doc_lim.empty() ? nullptr : (const int32_t *)(t + pl->off_d);
  Prologue pro;
  pro.links = lp.links;
  pro.reqs = lp.reqs;
  return launch_call(s, pl->C, lp, pl->work, pro, q, k_self, v_self, softmax_scale, out, lse,
                     (hipStream_t)stream);
}

pic_status pic_link_plan_destroy(pic_link_plan *pl) {
  if (!pl) return PIC_OK;
  if (pl->dev) {
    DeviceGuard dg(pl->store->device);
    (void)hipDeviceSynchronize();
    (void)hipFree(pl->dev);
  }
  for (uint64_t id : pl->C.P.ids) {
    auto it = pl->store->map.find(id);
    if (it != pl->store->map.end()) --it->second.plan_refs;
  }
  --pl->store->live_plans;
  delete pl;
  return PIC_OK;
}

pic_status pic_debug_gather(pic_store *s, const uint64_t *ids, int32_t n, int32_t layer,
                            void *k_out, void *v_out, void *stream) {
  if (!s) return fail(PIC_ERR_INVALID, "store is NULL");
  if (n < 0 || (n > 0 && !ids)) return fail(PIC_ERR_INVALID, "bad id list");
  if (layer < 0 || layer >= s->n_layers)
    return fail(PIC_ERR_INVALID, "layer %d outside the store's %d layers", layer, s->n_layers);
  const bool gqa = s->desc.kind == PIC_GQA;
  std::vector<LinkEntry> links;
  links.reserve(n);
  int64_t toks = 0;
  for (int32_t i = 0; i < n; ++i) {
    auto it = s->map.find(ids[i]);
    if (it == s->map.end()) return fail(PIC_ERR_NOT_FOUND, "chunk id 0x%llx not in the store",
                                        (unsigned long long)ids[i]);
    for (const Run &r : it->second.runs) {
      LinkEntry E = run_entry(s, r, layer);
      E.tile0 = 0;
      E.tok0 = (int32_t)toks;
      links.push_back(E);
      toks += r.ntok;
    }
  }
  n = (int32_t)links.size();
  if (toks == 0) return PIC_OK;
  if (!k_out || (gqa && !v_out)) return fail(PIC_ERR_INVALID, "k_out/v_out is NULL");
  if (!gqa && v_out) return fail(PIC_ERR_INVALID, "v_out must be NULL for MLA");
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(PIC_ERR_HIP, "cannot select the store's device");
  const hipStream_t st = (hipStream_t)stream;
  Stage *stage = nullptr;
  pic_status rc = stage_acquire(s, sizeof(LinkEntry) * n, &stage);
  if (rc != PIC_OK) return rc;
  memcpy(stage->host, links.data(), sizeof(LinkEntry) * n);
  HIP_TRY(launch_table_copy(stage->host_dev, stage->dev, (int64_t)(sizeof(LinkEntry) * n), st),
          "table_copy_kernel");
  const pic_store_desc &d = s->desc;
  hipError_t e = launch_gather((const LinkEntry *)stage->dev, n, toks, d.n_kv_heads,
                               d.d_k, d.d_v, !gqa, s->esz, k_out, v_out, st);
  if (e != hipSuccess) return hip_fail(e, "gather_kernel");
  HIP_TRY(hipEventRecord(stage->done, st), "hipEventRecord(stage)");
  stage->pending = true;
  return PIC_OK;
}

pic_status pic_debug_request_order(const int32_t *q_len, const int32_t *self_len,
                                   const int32_t *doc_tiles, int32_t batch, int32_t n_q_heads,
                                   int32_t n_kv_heads, int32_t cus, int32_t xcds,
                                   int32_t *order_out, double *finish_out) {
  if (batch < 0 || (batch > 0 && (!q_len || !self_len || !doc_tiles || !order_out)))
    return fail(PIC_ERR_INVALID, "NULL array");
  if (n_kv_heads <= 0 || n_q_heads <= 0 || n_q_heads % n_kv_heads || cus <= 0 || xcds <= 0 ||
      cus % xcds)
    return fail(PIC_ERR_INVALID, "bad head counts or device shape");
  Plan P;
  P.reqs.resize(batch);
  int32_t max_rows = 0;
  const int group = n_q_heads / n_kv_heads;
  for (int32_t r = 0; r < batch; ++r) {
    if (q_len[r] < 0 || self_len[r] < 0 || doc_tiles[r] < 0 ||
        (int64_t)q_len[r] * group > INT32_MAX / 2 || self_len[r] > INT32_MAX / 2 ||
        doc_tiles[r] > INT32_MAX / 4)
      return fail(PIC_ERR_INVALID, "request %d: length out of range", r);
    ReqEntry &R = P.reqs[r];
    R = ReqEntry{};
    R.lq = q_len[r];
    R.ls = self_len[r];
    R.doc_tiles = doc_tiles[r];
    R.tiles = R.doc_tiles + (R.ls + kTile - 1) / kTile;
    max_rows = std::max(max_rows, R.lq * group);
  }
  // heaviest first, as plan_call orders
  P.order.resize(batch);
  for (int32_t r = 0; r < batch; ++r) P.order[r] = r;
  std::stable_sort(P.order.begin(), P.order.end(), [&](int32_t a, int32_t b) {
    return (int64_t)P.reqs[a].tiles * P.reqs[a].lq > (int64_t)P.reqs[b].tiles * P.reqs[b].lq;
  });
  LinkParams lp{};
  lp.batch = batch;
  lp.n_q_heads = n_q_heads;
  lp.n_kv_heads = n_kv_heads;
  lp.group = group;
  lp.n_xcd = xcds;
  const int rows_per_block = mfma_d128_rows_per_block();
  lp.nrb = std::max(1, (max_rows + rows_per_block - 1) / rows_per_block);
  lp.n_groups = (int32_t)round_up((int64_t)batch * n_kv_heads, xcds);
  double finish[2];
  balance_order_d128(nullptr, P, lp, rows_per_block, cus / xcds * mfma_d128_blocks_per_cu(), finish);
  std::copy(P.order.begin(), P.order.end(), order_out);
  if (finish_out) {
    finish_out[0] = finish[0];
    finish_out[1] = finish[1];
  }
  return PIC_OK;
}

namespace {

// Shared checks of the two MLA projections: sizes, 16-byte aligned device
// buffers.
pic_status check_proj(int32_t n_tokens, int32_t n_heads, std::initializer_list<const void *> bufs) {
  if (n_tokens < 0 || n_heads <= 0 || n_heads > 1024)
    return fail(PIC_ERR_INVALID, "n_tokens must be >= 0 and n_heads 1..1024");
  if ((int64_t)n_tokens * n_heads > INT32_MAX / 4) return fail(PIC_ERR_INVALID, "too many rows");
  if (n_tokens == 0) return PIC_OK;
  for (const void *b : bufs) {
    if (!b) return fail(PIC_ERR_INVALID, "a tensor pointer is NULL");
    if ((uintptr_t)b % 16) return fail(PIC_ERR_INVALID, "tensors must be 16-byte aligned");
  }
  return PIC_OK;
}

}  // namespace

pic_status pic_mla_absorb_q(int32_t n_tokens, int32_t n_heads, const void *q, const void *w_uk_t,
                            void *q_out, void *stream) {
  pic_status rc = check_proj(n_tokens, n_heads, {q, w_uk_t, q_out});
  if (rc != PIC_OK || n_tokens == 0) return rc;
  hipError_t e = launch_mla_absorb_q(q, w_uk_t, q_out, n_tokens, n_heads, device_shape(),
                                     (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "proj_kernel (absorb)");
  return PIC_OK;
}

pic_status pic_mla_up_v(int32_t n_tokens, int32_t n_heads, const void *o_lat, const void *w_uv,
                        void *out, void *stream) {
  pic_status rc = check_proj(n_tokens, n_heads, {o_lat, w_uv, out});
  if (rc != PIC_OK || n_tokens == 0) return rc;
  hipError_t e = launch_mla_up_v(o_lat, w_uv, out, n_tokens, n_heads, device_shape(),
                                 (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "proj_kernel (up)");
  return PIC_OK;
}

pic_status pic_prof_begin_sampled(int32_t every) {
  if (every < 1 || every > 1000000) return fail(PIC_ERR_INVALID, "every must be 1..1000000");
  std::lock_guard<std::mutex> g(g_prof.mu);
  for (auto &ev : g_prof.events) g_prof.spare.push_back(ev);
  g_prof.events.clear();
  g_prof.every = every;
  g_prof.seen = 0;
  g_prof.on = true;
  return PIC_OK;
}

pic_status pic_prof_begin(void) { return pic_prof_begin_sampled(1); }

pic_status pic_prof_end(double *kernel_ms, int64_t *launches, char *name_buf, int32_t name_len) {
  std::lock_guard<std::mutex> g(g_prof.mu);
  g_prof.on = false;
  double total = 0.0;
  for (auto &ev : g_prof.events) {
    HIP_TRY(hipEventSynchronize(ev.second), "hipEventSynchronize(prof)");
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, ev.first, ev.second), "hipEventElapsedTime");
    total += ms;
  }
  if (kernel_ms) *kernel_ms = total;
  if (launches) *launches = (int64_t)g_prof.events.size();
  if (name_buf && name_len > 0) {
    snprintf(name_buf, (size_t)name_len, "%s", g_prof.name.c_str());
  }
  for (auto &ev : g_prof.events) g_prof.spare.push_back(ev);
  g_prof.events.clear();
  return PIC_OK;
}

// Times one launch of a peak microbenchmark on `stream` (blocking).
static pic_status time_peak(hipStream_t st, double *ms_out,
                            const std::function<hipError_t(float *)> &launch) {
  float *scratch = nullptr;
  HIP_TRY(hipMalloc(&scratch, (size_t)pic::peak_out_floats() * sizeof(float)), "hipMalloc(peak)");
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreateWithFlags(&e0, hipEventDisableSystemFence);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&e1, hipEventDisableSystemFence);
  if (e == hipSuccess) e = hipEventRecord(e0, st);
  if (e == hipSuccess) e = launch(scratch);
  if (e == hipSuccess) e = hipEventRecord(e1, st);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipFree(scratch);
  if (e != hipSuccess) return hip_fail(e, "peak microbenchmark");
  *ms_out = ms;
  return PIC_OK;
}

pic_status pic_peak_mfma_bf16(int32_t iters, double *tflops, void *stream) {
  if (!tflops) return fail(PIC_ERR_INVALID, "tflops is NULL");
  if (iters <= 0 || iters > (1 << 22)) return fail(PIC_ERR_INVALID, "iters must be 1..2^22");
  double ms = 0.0;
  const pic_status rc = time_peak((hipStream_t)stream, &ms, [&](float *out) {
    return pic::launch_peak_mfma(out, iters, (hipStream_t)stream);
  });
  if (rc != PIC_OK) return rc;
  *tflops = ms > 0.0 ? pic::peak_mfma_flops(iters) / (ms * 1e-3) / 1e12 : 0.0;
  return PIC_OK;
}

pic_status pic_peak_hbm_read(const void *buf, int64_t bytes, double *gbs, void *stream) {
  if (!gbs || !buf) return fail(PIC_ERR_INVALID, "buf and gbs must not be NULL");
  if (bytes <= 0 || bytes % 16 != 0 || (uintptr_t)buf % 16 != 0)
    return fail(PIC_ERR_INVALID, "bytes must be a positive multiple of 16 and buf 16-byte aligned");
  hipPointerAttribute_t at{};
  if (hipPointerGetAttributes(&at, buf) != hipSuccess || at.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(PIC_ERR_INVALID, "buf is not device memory");
  }
  double ms = 0.0;
  const pic_status rc = time_peak((hipStream_t)stream, &ms, [&](float *out) {
    return pic::launch_peak_read(buf, bytes, out, (hipStream_t)stream);
  });
  if (rc != PIC_OK) return rc;
  *gbs = ms > 0.0 ? (double)bytes / (ms * 1e-3) / 1e9 : 0.0;
  return PIC_OK;
}

pic_status pic_peak_hbm_write(void *buf, int64_t bytes, double *gbs, void *stream) {
  if (!gbs || !buf) return fail(PIC_ERR_INVALID, "buf and gbs must not be NULL");
  if (bytes <= 0 || bytes % 16 != 0 || (uintptr_t)buf % 16 != 0)
    return fail(PIC_ERR_INVALID, "bytes must be a positive multiple of 16 and buf 16-byte aligned");
  hipPointerAttribute_t at{};
  if (hipPointerGetAttributes(&at, buf) != hipSuccess || at.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return fail(PIC_ERR_INVALID, "buf is not device memory");
  }
  double ms = 0.0;
  const pic_status rc = time_peak((hipStream_t)stream, &ms, [&](float *) {
    return pic::launch_peak_write(buf, bytes, (hipStream_t)stream);
  });
  if (rc != PIC_OK) return rc;
  *gbs = ms > 0.0 ? (double)bytes / (ms * 1e-3) / 1e9 : 0.0;
  return PIC_OK;
}

const char *pic_status_str(pic_status st) {
  switch (st) {
    case PIC_OK: return "PIC_OK";
    case PIC_ERR_INVALID: return "PIC_ERR_INVALID";
    case PIC_ERR_NOT_FOUND: return "PIC_ERR_NOT_FOUND";
    case PIC_ERR_EXISTS: return "PIC_ERR_EXISTS";
    case PIC_ERR_OOM: return "PIC_ERR_OOM";
    case PIC_ERR_HIP: return "PIC_ERR_HIP";
    case PIC_ERR_UNSUPPORTED: return "PIC_ERR_UNSUPPORTED";
  }
  return "PIC_ERR_?";
}

const char *pic_last_error(void) { return g_err.c_str(); }

}  // extern "C"
