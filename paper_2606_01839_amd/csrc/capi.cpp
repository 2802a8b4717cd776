// C ABI of the library (declared in include/conserve_attn.h): argument validation, host metadata
// (pages, conversations, plans), metadata upload through a pinned ring, kernel launches.
#include "conserve_attn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include "host/host_state.hpp"
#include "kernels.hpp"

namespace {

thread_local std::string g_err;

cs_status fail(cs_status code, const std::string& msg) {
  g_err = msg;
  return code;
}

constexpr size_t kAlign = 256;
constexpr size_t kRingBytes = size_t(8) << 20;  // metadata ring (device + pinned host), 4 quarters
constexpr size_t kQuarter = kRingBytes / 4;
constexpr int kMinSplit = 128;                   // smallest decode split: bounds the partials
// Splits (waves) a decode launch aims for (16 per CU). Half as many (longer splits, fewer items to
// merge) made the 32-layer mixed trace 5% slower, twice as many 1% slower.
constexpr int64_t kDecodeTargetItems = 4096;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct WsLayout {
  size_t page_table, partials, partials2, ring, total;
  size_t partial_floats;
};

int64_t max_decode_items(const cs_pool_desc& d) {
  // sum_b ceil(L_b / kMinSplit) <= total tokens / kMinSplit + batch
  return d.n_pages * cs::kPage / kMinSplit + d.max_convs;
}

WsLayout ws_layout(const cs_pool_desc& d) {
  WsLayout w{};
  const int group = d.n_q_heads / d.n_kv_heads;
  w.page_table = 0;
  size_t pt_bytes = static_cast<size_t>(d.max_convs) * static_cast<size_t>(d.max_pages_per_conv) * 4;
  w.partials = align_up(pt_bytes, kAlign);
  w.partial_floats =
      static_cast<size_t>(max_decode_items(d)) * d.n_kv_heads * group * cs::partial_floats(d.head_dim);
  // A multi-layer pool gets a second partial buffer: cs_mixed_step merges layer l while it splits
  // layer l+1 in the same launch.
  w.partials2 = align_up(w.partials + w.partial_floats * 4, kAlign);
  const size_t second = d.n_layers > 1 ? w.partial_floats * 4 : 0;
  w.ring = align_up(w.partials2 + second, kAlign);
  w.total = w.ring + kRingBytes;
  return w;
}

const char* desc_problem(const cs_pool_desc* d) {
  if (!d) return "null descriptor";
  if (d->n_layers < 1) return "n_layers must be >= 1";
  if (d->n_kv_heads < 1 || d->n_q_heads < 1 || d->n_q_heads % d->n_kv_heads != 0)
    return "n_q_heads must be a positive multiple of n_kv_heads";
  const int group = d->n_q_heads / d->n_kv_heads;
  if (d->head_dim != 64 && d->head_dim != 128) return "head_dim must be 64 or 128";
  if (group != 1 && group != 2 && group != 4 && group != 8)
    return "n_q_heads/n_kv_heads must be 1, 2, 4 or 8";
  if (d->max_convs < 1 || d->max_convs > (1 << cs::ConvTable::kSlotBits))
    return "max_convs must be in [1, 2^20]";
  if (d->max_pages_per_conv < 1 || d->max_pages_per_conv > (1 << 26))
    return "max_pages_per_conv must be in [1, 2^26]";
  if (d->n_pages < 1 || d->n_pages > INT32_MAX) return "n_pages must be in [1, 2^31)";
  return nullptr;
}

}  // namespace

struct cs_pool {
  cs_pool_desc desc;
  char* kv;
  size_t kv_bytes;
  char* ws;
  size_t ws_bytes;
  WsLayout lay;
  cs::PagePool pages;
  cs::ConvTable convs;
  // device resources, created on first use
  bool dev_ready = false;
  int device = -1;
  char* h_ring = nullptr;
  size_t ring_head = 0;
  int cur_quarter = -1;
  hipEvent_t quarter_ev[4] = {};
  bool quarter_used[4] = {};
  hipEvent_t switch_ev = nullptr;
  hipStream_t stream = nullptr;
  bool have_stream = false;
  // second stream of cs_mixed_step (extend chunks run on it concurrently with the decode batch)
  hipStream_t side = nullptr;
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  // instrumentation: timing events around each kernel launch while enabled
  struct ProfEvent {
    hipEvent_t start, stop;
    int kind;
    int launches;
  };
  bool prof_on = false;
  int64_t fail_after = -1;  // cs_debug_fail_launches: launches left before the injected failure
  // an open span: one pair of events brackets a run of launches of one kind on one stream
  bool span_open = false;
  hipEvent_t span_start = nullptr;
  hipStream_t span_stream = nullptr;
  int span_kind = 0, span_launches = 0;
  std::vector<hipEvent_t> ev_free;
  std::vector<ProfEvent> prof_events;

  cs_pool(const cs_pool_desc& d, char* kvp, size_t kvb, char* wsp, size_t wsb, uint64_t seed)
      : desc(d), kv(kvp), kv_bytes(kvb), ws(wsp), ws_bytes(wsb), lay(ws_layout(d)),
        pages(d.n_pages, seed), convs(d.max_convs, d.max_pages_per_conv) {}

  cs::PoolGeom geom() const {
    cs::PoolGeom g;
    g.pool = kv;
    g.n_pages = desc.n_pages;
    g.n_layers = desc.n_layers;
    g.n_kv_heads = desc.n_kv_heads;
    g.n_q_heads = desc.n_q_heads;
    g.head_dim = desc.head_dim;
    g.page_table = reinterpret_cast<int32_t*>(ws + lay.page_table);
    g.max_pages = desc.max_pages_per_conv;
    return g;
  }
  float* partials() const { return reinterpret_cast<float*>(ws + lay.partials); }
  float* partials2() const { return reinterpret_cast<float*>(ws + lay.partials2); }
};

namespace {

cs_status hip_fail(hipError_t e, const char* what) {
  return fail(CS_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define CS_HIP(call, what)                        \
  do {                                            \
    hipError_t e_ = (call);                       \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

cs_status ensure_device(cs_pool* p) {
  if (p->dev_ready) return CS_OK;
  int dev = 0;
  CS_HIP(hipGetDevice(&dev), "hipGetDevice");
  void* h = nullptr;
  CS_HIP(hipHostMalloc(&h, kRingBytes, hipHostMallocDefault), "hipHostMalloc(metadata ring)");
  for (int i = 0; i < 4; ++i) {
    hipError_t e = hipEventCreateWithFlags(&p->quarter_ev[i], hipEventDisableTiming);
    if (e != hipSuccess) {
      for (int k = 0; k < i; ++k) (void)hipEventDestroy(p->quarter_ev[k]);
      (void)hipHostFree(h);
      return hip_fail(e, "hipEventCreate");
    }
  }
  hipError_t e = hipEventCreateWithFlags(&p->switch_ev, hipEventDisableTiming);
  if (e != hipSuccess) {
    for (int k = 0; k < 4; ++k) (void)hipEventDestroy(p->quarter_ev[k]);
    (void)hipHostFree(h);
    return hip_fail(e, "hipEventCreate");
  }
  p->h_ring = static_cast<char*>(h);
  p->device = dev;
  p->dev_ready = true;
  return CS_OK;
}

// All of a pool's work is chained on one stream at a time; a new stream first waits for the old.
cs_status use_stream(cs_pool* p, hipStream_t s) {
  if (p->have_stream && s != p->stream) {
    CS_HIP(hipEventRecord(p->switch_ev, p->stream), "hipEventRecord");
    CS_HIP(hipStreamWaitEvent(s, p->switch_ev, 0), "hipStreamWaitEvent");
  }
  p->stream = s;
  p->have_stream = true;
  return CS_OK;
}

hipError_t take_event(cs_pool* p, hipEvent_t* e) {
  if (!p->ev_free.empty()) {
    *e = p->ev_free.back();
    p->ev_free.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(e);
}

// Launch a kernel on stream `s`; while profiling, bracket it with timing events on that stream
// (inside an open span the span's events cover it and it only counts as one more launch).
template <typename F>
cs_status timed_launch_on(cs_pool* p, hipStream_t s, int kind, const char* what, F&& launch) {
  if (p->fail_after == 0) return fail(CS_EHIP, std::string(what) + ": failure injected by cs_debug_fail_launches");
  if (p->fail_after > 0) --p->fail_after;
  if (p->prof_on && p->span_open) {
    CS_HIP(launch(), what);
    ++p->span_launches;
    return CS_OK;
  }
  hipEvent_t a = nullptr, b = nullptr;
  if (p->prof_on) {
    CS_HIP(take_event(p, &a), "hipEventCreate");
    CS_HIP(take_event(p, &b), "hipEventCreate");
    CS_HIP(hipEventRecord(a, s), "hipEventRecord");
  }
  CS_HIP(launch(), what);
  if (p->prof_on) {
    CS_HIP(hipEventRecord(b, s), "hipEventRecord");
    p->prof_events.push_back({a, b, kind, 1});
  }
  return CS_OK;
}

// Open a timing span of `kind` on stream `s` (no-op while profiling is off). A run of launches
// then records two events in all instead of two per launch, which keeps the instrumentation's own
// cost out of multi-layer steps; the span's time includes the short gaps between its launches.
cs_status span_begin(cs_pool* p, hipStream_t s, int kind) {
  if (!p->prof_on) return CS_OK;
  hipEvent_t a = nullptr;
  CS_HIP(take_event(p, &a), "hipEventCreate");
  const hipError_t e = hipEventRecord(a, s);
  if (e != hipSuccess) {
    p->ev_free.push_back(a);
    return hip_fail(e, "hipEventRecord");
  }
  p->span_start = a;
  p->span_open = true;
  p->span_stream = s;
  p->span_kind = kind;
  p->span_launches = 0;
  return CS_OK;
}

// Close the open span (no-op if none is open); called on error paths too.
cs_status span_end(cs_pool* p) {
  if (!p->span_open) return CS_OK;
  p->span_open = false;
  hipEvent_t b = nullptr;
  hipError_t e = take_event(p, &b);
  if (e == hipSuccess) {
    e = hipEventRecord(b, p->span_stream);
    if (e != hipSuccess) p->ev_free.push_back(b);
  }
  if (e != hipSuccess) {
    p->ev_free.push_back(p->span_start);
    return hip_fail(e, "hipEventRecord");
  }
  p->prof_events.push_back({p->span_start, b, p->span_kind, p->span_launches});
  return CS_OK;
}

template <typename F>
cs_status timed_launch(cs_pool* p, int kind, const char* what, F&& launch) {
  return timed_launch_on(p, p->stream, kind, what, launch);
}

// The second stream and its fork/join events, created on first use.
cs_status ensure_side(cs_pool* p) {
  if (p->side) return CS_OK;
  hipStream_t s = nullptr;
  CS_HIP(hipStreamCreateWithFlags(&s, hipStreamNonBlocking), "hipStreamCreate");
  hipEvent_t f = nullptr, j = nullptr;
  hipError_t e = hipEventCreateWithFlags(&f, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&j, hipEventDisableTiming);
  if (e != hipSuccess) {
    if (f) (void)hipEventDestroy(f);
    (void)hipStreamDestroy(s);
    return hip_fail(e, "hipEventCreate");
  }
  p->side = s;
  p->fork_ev = f;
  p->join_ev = j;
  return CS_OK;
}

// Reserve `n` bytes of the metadata ring inside one quarter. Entering a quarter records an event
// closing the previous one (everything enqueued so far) and waits for the event that closed the
// entered quarter last time round, so a region is never rewritten while a copy or kernel of an
// earlier call may still read it.
cs_status ring_reserve(cs_pool* p, size_t n, size_t* off_out) {
  n = align_up(std::max<size_t>(n, 1), kAlign);
  if (n > kQuarter) return fail(CS_ENOMEM, "metadata for one launch exceeds the upload ring");
  size_t off = p->ring_head;
  if (off / kQuarter != (off + n - 1) / kQuarter || off + n > kRingBytes)
    off = ((off + kQuarter - 1) / kQuarter) * kQuarter;
  if (off + n > kRingBytes) off = 0;
  const int q = static_cast<int>(off / kQuarter);
  if (q != p->cur_quarter) {
    if (p->cur_quarter >= 0) {
      CS_HIP(hipEventRecord(p->quarter_ev[p->cur_quarter], p->stream), "hipEventRecord");
      p->quarter_used[p->cur_quarter] = true;
    }
    if (p->quarter_used[q]) CS_HIP(hipEventSynchronize(p->quarter_ev[q]), "hipEventSynchronize");
    p->cur_quarter = q;
  }
  p->ring_head = off + n;
  *off_out = off;
  return CS_OK;
}

// Copy host bytes into the ring and enqueue their upload; returns the device address.
cs_status upload(cs_pool* p, const void* src, size_t n, void** dev_out) {
  size_t off = 0;
  cs_status st = ring_reserve(p, n, &off);
  if (st != CS_OK) return st;
  std::memcpy(p->h_ring + off, src, n);
  char* d = p->ws + p->lay.ring + off;
  CS_HIP(hipMemcpyAsync(d, p->h_ring + off, n, hipMemcpyHostToDevice, p->stream), "hipMemcpyAsync");
  *dev_out = d;
  return CS_OK;
}

// Two host arrays uploaded back to back in one reservation.
template <typename A, typename B>
cs_status upload2(cs_pool* p, const std::vector<A>& a, const std::vector<B>& b, A** da, B** db) {
  const size_t na = align_up(a.size() * sizeof(A), 16), nb = b.size() * sizeof(B);
  size_t off = 0;
  cs_status st = ring_reserve(p, na + nb, &off);
  if (st != CS_OK) return st;
  if (!a.empty()) std::memcpy(p->h_ring + off, a.data(), a.size() * sizeof(A));
  if (!b.empty()) std::memcpy(p->h_ring + off + na, b.data(), nb);
  char* d = p->ws + p->lay.ring + off;
  CS_HIP(hipMemcpyAsync(d, p->h_ring + off, na + nb, hipMemcpyHostToDevice, p->stream),
         "hipMemcpyAsync");
  *da = reinterpret_cast<A*>(d);
  *db = reinterpret_cast<B*>(d + na);
  return CS_OK;
}

cs_status check_convs(const cs_pool* p, int32_t n, const cs_conv* convs, std::vector<const cs::Conv*>& out) {
  if (n < 0) return fail(CS_EINVAL, "negative batch size");
  if (n > 0 && !convs) return fail(CS_EINVAL, "null conversation array");
  out.clear();
  std::unordered_set<int32_t> seen;
  for (int32_t i = 0; i < n; ++i) {
    const cs::Conv* c = p->convs.find(convs[i]);
    if (!c) return fail(CS_ENOENT, "unknown conversation handle " + std::to_string(convs[i]));
    if (!seen.insert(convs[i]).second)
      return fail(CS_EINVAL, "conversation " + std::to_string(convs[i]) + " appears twice in a batch");
    out.push_back(c);
  }
  return CS_OK;
}

size_t wire_size(const cs_pool_desc& d, int64_t len) {
  return static_cast<size_t>(d.n_layers) * static_cast<size_t>(cs::pages_for(len)) *
         static_cast<size_t>(d.n_kv_heads) * 2 * cs::kPage * static_cast<size_t>(d.head_dim) * 2;
}

hipStream_t as_stream(cs_stream s) { return reinterpret_cast<hipStream_t>(s); }

// Extend/prefill work uploaded once and launchable for any layer.
struct ExtendWork {
  struct Part {
    cs::ExtendConvDesc* convs;
    cs::ExtendTile* tiles;
    int n_tiles;
  };
  std::vector<Part> parts;
};

cs_status upload_extend(cs_pool* p, const std::vector<int32_t>& slots, const std::vector<int64_t>& lens,
                        const std::vector<int32_t>& q_lens, ExtendWork* w) {
  const int tile = cs::extend_query_tile(p->desc.head_dim, p->desc.n_q_heads / p->desc.n_kv_heads);
  cs::ExtendPlan plan = cs::plan_extend(slots, lens, q_lens, tile);
  const size_t desc_bytes = align_up(plan.convs.size() * sizeof(cs::ExtendConvDesc), 16);
  if (desc_bytes + kAlign + sizeof(cs::ExtendTile) > kQuarter)
    return fail(CS_ENOMEM, "batch descriptor exceeds the metadata ring");
  const size_t max_tiles = (kQuarter - desc_bytes - kAlign) / sizeof(cs::ExtendTile);
  for (size_t t0 = 0; t0 < plan.tiles.size(); t0 += max_tiles) {
    const size_t t1 = std::min(plan.tiles.size(), t0 + max_tiles);
    std::vector<cs::ExtendTile> part(plan.tiles.begin() + t0, plan.tiles.begin() + t1);
    ExtendWork::Part pw{nullptr, nullptr, static_cast<int>(part.size())};
    cs_status st = upload2(p, plan.convs, part, &pw.convs, &pw.tiles);
    if (st != CS_OK) return st;
    w->parts.push_back(pw);
  }
  return CS_OK;
}

cs_status launch_extend_layer(cs_pool* p, const ExtendWork& w, int layer, const void* q, void* out,
                              hipStream_t s) {
  const cs::PoolGeom g = p->geom();
  for (const auto& pw : w.parts) {
    cs_status st = timed_launch_on(p, s, CS_PROF_ATTN_FWD, "attention launch", [&] {
      return cs::launch_extend(g, layer, pw.convs, pw.tiles, pw.n_tiles, q, out, s);
    });
    if (st != CS_OK) return st;
  }
  return CS_OK;
}

struct DecodeWork {
  cs::DecodeConvDesc* convs = nullptr;
  int32_t* order = nullptr;  // launch order of the items
  int n_convs = 0, n_items = 0, split = 0;
  bool single = false;  // one work item per conversation: the split writes the output directly
};

cs::DecodePlan plan_decode_batch(const cs_pool* p, const std::vector<int32_t>& slots,
                                 const std::vector<int64_t>& lens) {
  return cs::plan_decode(slots, lens, p->desc.n_kv_heads, kDecodeTargetItems);
}

// Descriptors and launch order of a decode plan, as uploaded back to back.
size_t decode_upload_bytes(const cs::DecodePlan& plan) {
  return align_up(plan.convs.size() * sizeof(cs::DecodeConvDesc), 16) + plan.order.size() * sizeof(int32_t);
}

cs_status check_decode_plan(const cs_pool* p, const cs::DecodePlan& plan) {
  if (plan.n_items > max_decode_items(p->desc)) return fail(CS_ENOMEM, "decode partials exceed the workspace");
  if (decode_upload_bytes(plan) > kQuarter) return fail(CS_ENOMEM, "batch descriptor exceeds the metadata ring");
  return CS_OK;
}

cs_status upload_decode(cs_pool* p, const cs::DecodePlan& plan, DecodeWork* w) {
  cs_status st = check_decode_plan(p, plan);
  if (st != CS_OK) return st;
  if ((st = upload2(p, plan.convs, plan.order, &w->convs, &w->order)) != CS_OK) return st;
  w->n_convs = static_cast<int>(plan.convs.size());
  w->n_items = plan.n_items;
  w->split = plan.split_tokens;
  w->single = plan.single_item;
  return CS_OK;
}

// Split, then merge; when every conversation is one work item the split writes the output itself.
cs_status launch_decode_layer(cs_pool* p, const DecodeWork& w, int layer, const void* q, void* out) {
  const cs::PoolGeom g = p->geom();
  cs_status st = timed_launch(p, CS_PROF_DECODE_SPLIT, "decode split launch", [&] {
    return cs::launch_decode_split(g, layer, w.convs, w.order, w.n_convs, w.n_items, w.split, q, p->partials(),
                                   w.single ? out : nullptr, p->stream);
  });
  if (st != CS_OK || w.single) return st;
  return timed_launch(p, CS_PROF_DECODE_MERGE, "decode merge launch", [&] {
    return cs::launch_decode_merge(g, w.convs, w.n_convs, p->partials(), out, p->stream);
  });
}

cs_status attend(cs_pool* p, int32_t n, const cs_conv* convs, const int32_t* q_lens, int32_t layer,
                 const void* q, void* out, cs_stream stream, bool turn1) {
  if (!p) return fail(CS_EINVAL, "null pool");
  std::vector<const cs::Conv*> cv;
  cs_status st = check_convs(p, n, convs, cv);
  if (st != CS_OK) return st;
  if (n > 0 && !q_lens) return fail(CS_EINVAL, "null q_lens");
  if (layer < 0 || layer >= p->desc.n_layers) return fail(CS_ERANGE, "layer out of range");
  int64_t rows = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (q_lens[i] < 0) return fail(CS_EINVAL, "negative q_len");
    if (q_lens[i] > cv[i]->len)
      return fail(CS_ESTATE, "q_len " + std::to_string(q_lens[i]) + " exceeds conversation length " +
                                 std::to_string(cv[i]->len));
    if (turn1 && q_lens[i] != cv[i]->len)
      return fail(CS_ESTATE, "turn-1 prefill needs q_len == conversation length (append the prompt first)");
    rows += q_lens[i];
  }
  if (rows == 0) return CS_OK;
  if (rows > INT32_MAX) return fail(CS_EINVAL, "too many query rows");
  if (!q || !out) return fail(CS_EINVAL, "null q/out");
  if ((st = ensure_device(p)) != CS_OK) return st;
  if ((st = use_stream(p, as_stream(stream))) != CS_OK) return st;

  std::vector<int32_t> slots(n), ql(q_lens, q_lens + n);
  std::vector<int64_t> lens(n);
  for (int32_t i = 0; i < n; ++i) {
    slots[i] = cs::ConvTable::slot_of(convs[i]);
    lens[i] = cv[i]->len;
  }
  ExtendWork w;
  if ((st = upload_extend(p, slots, lens, ql, &w)) != CS_OK) return st;
  return launch_extend_layer(p, w, layer, q, out, p->stream);
}

cs_status append_impl(cs_pool* p, int32_t n, const cs_conv* convs, const int32_t* n_new,
                      const void* k, const void* v, cs_stream stream) {
  if (!p) return fail(CS_EINVAL, "null pool");
  std::vector<const cs::Conv*> cv;
  cs_status st = check_convs(p, n, convs, cv);
  if (st != CS_OK) return st;
  if (n > 0 && !n_new) return fail(CS_EINVAL, "null n_new");
  int64_t total = 0, need_pages = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (n_new[i] < 0) return fail(CS_EINVAL, "negative token count");
    const int64_t nl = cv[i]->len + n_new[i];
    if (cs::pages_for(nl) > p->desc.max_pages_per_conv)
      return fail(CS_ERANGE, "conversation would exceed max_pages_per_conv");
    need_pages += cs::pages_for(nl) - cs::pages_for(cv[i]->len);
    total += n_new[i];
  }
  if (total == 0) return CS_OK;
  if (total > INT32_MAX) return fail(CS_EINVAL, "too many tokens in one append");
  if (!k || !v) return fail(CS_EINVAL, "null k/v");
  if (need_pages > p->pages.free_count())
    return fail(CS_ENOMEM, "KV pool exhausted: need " + std::to_string(need_pages) + " pages, " +
                               std::to_string(p->pages.free_count()) + " free");
  if ((st = ensure_device(p)) != CS_OK) return st;
  if ((st = use_stream(p, as_stream(stream))) != CS_OK) return st;

  // Reserve pages (cannot fail now) and build the chunks; lengths are committed only after every
  // upload and launch has been issued. If one of those fails, the reserved pages go back to the
  // free list in their old order and nothing about the conversations changes. (Launches already
  // issued may have written the new tokens into the reserved pages and into unused slots past a
  // conversation's end; no kernel reads those: attention masks keys past the length, pack writes
  // zeros there, and the pages return to the free list.)
  std::vector<int32_t> slots(n), nn(n_new, n_new + n);
  std::vector<int64_t> old_lens(n);
  std::vector<size_t> old_pages(n);
  std::vector<const std::vector<int32_t>*> lists(n);
  for (int32_t i = 0; i < n; ++i) {
    cs::Conv* c = p->convs.find(convs[i]);
    slots[i] = cs::ConvTable::slot_of(convs[i]);
    old_lens[i] = c->len;
    old_pages[i] = c->pages.size();
    p->pages.alloc(cs::pages_for(c->len + n_new[i]) - cs::pages_for(c->len), c->pages);
    lists[i] = &c->pages;
  }
  std::vector<cs::PageChunk> chunks = cs::plan_append(slots, old_lens, nn, lists);
  auto roll_back = [&] {
    std::vector<int32_t> taken;
    for (int32_t i = 0; i < n; ++i) {
      cs::Conv* c = p->convs.find(convs[i]);
      taken.insert(taken.end(), c->pages.begin() + static_cast<std::ptrdiff_t>(old_pages[i]), c->pages.end());
      c->pages.resize(old_pages[i]);
    }
    p->pages.unalloc(taken);
  };

  const cs::PoolGeom g = p->geom();
  const size_t per = kQuarter / sizeof(cs::PageChunk) - 1;
  for (size_t c0 = 0; c0 < chunks.size(); c0 += per) {
    const size_t c1 = std::min(chunks.size(), c0 + per);
    void* d = nullptr;
    st = upload(p, chunks.data() + c0, (c1 - c0) * sizeof(cs::PageChunk), &d);
    if (st == CS_OK)
      st = timed_launch(p, CS_PROF_APPEND, "append launch", [&] {
        return cs::launch_append(g, static_cast<const cs::PageChunk*>(d), static_cast<int>(c1 - c0), k, v,
                                 total, p->stream);
      });
    if (st != CS_OK) {
      roll_back();
      return st;
    }
  }
  for (int32_t i = 0; i < n; ++i) p->convs.find(convs[i])->len += n_new[i];
  return CS_OK;
}

}  // namespace

extern "C" {

const char* cs_last_error(void) { return g_err.c_str(); }

size_t cs_pool_kv_bytes(const cs_pool_desc* d) {
  if (desc_problem(d)) return 0;
  return static_cast<size_t>(d->n_layers) * static_cast<size_t>(d->n_pages) *
         static_cast<size_t>(d->n_kv_heads) * 2 * cs::kPage * static_cast<size_t>(d->head_dim) * 2;
}

size_t cs_pool_workspace_bytes(const cs_pool_desc* d) {
  if (desc_problem(d)) return 0;
  return ws_layout(*d).total;
}

cs_status cs_pool_create(const cs_pool_desc* d, void* kv_base, size_t kv_bytes, void* ws_base,
                         size_t ws_bytes, uint64_t seed, cs_pool** out) {
  if (const char* why = desc_problem(d)) return fail(CS_EINVAL, why);
  if (!out) return fail(CS_EINVAL, "null out");
  if (!kv_base || !ws_base) return fail(CS_EINVAL, "null kv or workspace base");
  if (reinterpret_cast<uintptr_t>(kv_base) % kAlign || reinterpret_cast<uintptr_t>(ws_base) % kAlign)
    return fail(CS_EINVAL, "kv and workspace bases must be 256-byte aligned");
  if (kv_bytes < cs_pool_kv_bytes(d)) return fail(CS_EINVAL, "kv buffer smaller than cs_pool_kv_bytes");
  if (ws_bytes < cs_pool_workspace_bytes(d))
    return fail(CS_EINVAL, "workspace smaller than cs_pool_workspace_bytes");
  cs_pool* p = new (std::nothrow)
      cs_pool(*d, static_cast<char*>(kv_base), kv_bytes, static_cast<char*>(ws_base), ws_bytes, seed);
  if (!p) return fail(CS_ENOMEM, "host allocation failed");
  *out = p;
  return CS_OK;
}

cs_status cs_pool_destroy(cs_pool* p) {
  if (!p) return fail(CS_EINVAL, "null pool");
  cs_status st = CS_OK;
  if (p->dev_ready) {
    if (p->have_stream && hipStreamSynchronize(p->stream) != hipSuccess)
      st = fail(CS_EHIP, "hipStreamSynchronize failed while destroying the pool");
    for (auto& e : p->quarter_ev) (void)hipEventDestroy(e);
    for (auto& e : p->ev_free) (void)hipEventDestroy(e);
    for (auto& pe : p->prof_events) {
      (void)hipEventDestroy(pe.start);
      (void)hipEventDestroy(pe.stop);
    }
    (void)hipEventDestroy(p->switch_ev);
    if (p->side) {
      if (hipStreamSynchronize(p->side) != hipSuccess)
        st = fail(CS_EHIP, "hipStreamSynchronize failed while destroying the pool");
      (void)hipEventDestroy(p->fork_ev);
      (void)hipEventDestroy(p->join_ev);
      (void)hipStreamDestroy(p->side);
    }
    (void)hipHostFree(p->h_ring);
  }
  delete p;
  return st;
}

cs_status cs_pool_occupancy(const cs_pool* p, int64_t* used, int64_t* free_pages) {
  if (!p || !used || !free_pages) return fail(CS_EINVAL, "null argument");
  *used = p->pages.used_count();
  *free_pages = p->pages.free_count();
  return CS_OK;
}

cs_status cs_conv_create(cs_pool* p, cs_conv* out) {
  if (!p || !out) return fail(CS_EINVAL, "null argument");
  if (!p->convs.create(out)) return fail(CS_ENOMEM, "all conversation slots are live");
  return CS_OK;
}

cs_status cs_conv_destroy(cs_pool* p, cs_conv conv) {
  if (!p) return fail(CS_EINVAL, "null pool");
  if (!p->convs.find(conv)) return fail(CS_ENOENT, "unknown conversation handle");
  p->convs.destroy(conv, p->pages);
  return CS_OK;
}

cs_status cs_conv_len(const cs_pool* p, cs_conv conv, int64_t* tokens) {
  if (!p || !tokens) return fail(CS_EINVAL, "null argument");
  const cs::Conv* c = p->convs.find(conv);
  if (!c) return fail(CS_ENOENT, "unknown conversation handle");
  *tokens = c->len;
  return CS_OK;
}

cs_status cs_conv_pages(const cs_pool* p, cs_conv conv, int32_t* out, int64_t cap, int64_t* n) {
  if (!p || !n) return fail(CS_EINVAL, "null argument");
  const cs::Conv* c = p->convs.find(conv);
  if (!c) return fail(CS_ENOENT, "unknown conversation handle");
  *n = static_cast<int64_t>(c->pages.size());
  if (cap < *n) return fail(CS_ERANGE, "output capacity smaller than the page count");
  if (*n > 0 && !out) return fail(CS_EINVAL, "null output");
  std::copy(c->pages.begin(), c->pages.end(), out);
  return CS_OK;
}

cs_status cs_kv_append(cs_pool* p, cs_conv conv, int32_t n_new, const void* k, const void* v,
                       cs_stream stream) {
  return append_impl(p, 1, &conv, &n_new, k, v, stream);
}

cs_status cs_kv_append_batch(cs_pool* p, int32_t n_convs, const cs_conv* convs, const int32_t* n_new,
                             const void* k, const void* v, cs_stream stream) {
  return append_impl(p, n_convs, convs, n_new, k, v, stream);
}

cs_status cs_attn_prefill_turn1(cs_pool* p, int32_t n, const cs_conv* convs, const int32_t* q_lens,
                                int32_t layer, const void* q, void* out, cs_stream stream) {
  return attend(p, n, convs, q_lens, layer, q, out, stream, true);
}

cs_status cs_attn_extend(cs_pool* p, int32_t n, const cs_conv* convs, const int32_t* q_lens,
                         int32_t layer, const void* q, void* out, cs_stream stream) {
  return attend(p, n, convs, q_lens, layer, q, out, stream, false);
}

cs_status cs_attn_decode_batch(cs_pool* p, int32_t n, const cs_conv* convs, int32_t layer,
                               const void* q, void* out, cs_stream stream) {
  if (!p) return fail(CS_EINVAL, "null pool");
  std::vector<const cs::Conv*> cv;
  cs_status st = check_convs(p, n, convs, cv);
  if (st != CS_OK) return st;
  if (layer < 0 || layer >= p->desc.n_layers) return fail(CS_ERANGE, "layer out of range");
  for (int32_t i = 0; i < n; ++i)
    if (cv[i]->len < 1) return fail(CS_ESTATE, "decode on an empty conversation");
  if (n == 0) return CS_OK;
  if (!q || !out) return fail(CS_EINVAL, "null q/out");
  if ((st = ensure_device(p)) != CS_OK) return st;
  if ((st = use_stream(p, as_stream(stream))) != CS_OK) return st;
  std::vector<int32_t> slots(n);
  std::vector<int64_t> lens(n);
  for (int32_t i = 0; i < n; ++i) {
    slots[i] = cs::ConvTable::slot_of(convs[i]);
    lens[i] = cv[i]->len;
  }
  DecodeWork w;
  if ((st = upload_decode(p, plan_decode_batch(p, slots, lens), &w)) != CS_OK) return st;
  return launch_decode_layer(p, w, layer, q, out);
}

cs_status cs_attn_decode_batch_noalloc(cs_pool* p, int32_t n, const cs_conv* convs, int32_t layer,
                                       const void* q, void* out, cs_stream stream) {
  if (!p) return fail(CS_EINVAL, "null pool");
  std::vector<const cs::Conv*> cv;
  cs_status st = check_convs(p, n, convs, cv);
  if (st != CS_OK) return st;
  if (layer < 0 || layer >= p->desc.n_layers) return fail(CS_ERANGE, "layer out of range");
  for (int32_t i = 0; i < n; ++i)
    if (cv[i]->len < 1) return fail(CS_ESTATE, "decode on an empty conversation");
  if (n == 0) return CS_OK;
  if (!q || !out) return fail(CS_EINVAL, "null q/out");
  // The pool's device state (metadata ring) is created by its first device call, which allocates;
  // every pool holding a non-empty conversation has made one (an append or an unpack).
  if (!p->dev_ready) return fail(CS_ESTATE, "pool has no device state yet (no append or unpack ran)");
  int dev = -1;
  CS_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev != p->device) return fail(CS_EINVAL, "the current device is not the pool's device");
  std::vector<int32_t> slots(n);
  std::vector<int64_t> lens(n);
  for (int32_t i = 0; i < n; ++i) {
    slots[i] = cs::ConvTable::slot_of(convs[i]);
    lens[i] = cv[i]->len;
  }
  const cs::DecodePlan plan = plan_decode_batch(p, slots, lens);
  const size_t need = plan.single_item ? 0
      : static_cast<size_t>(plan.n_items) * p->desc.n_q_heads * cs::partial_floats(p->desc.head_dim);
  if (need > cs::kStaticScratchFloats)
    return fail(CS_ENOMEM, "decode partials (" + std::to_string(need * 4) + " bytes) exceed the " +
                               std::to_string(cs::kStaticScratchFloats * 4) + "-byte static scratch");
  if (decode_upload_bytes(plan) > kQuarter) return fail(CS_ENOMEM, "batch descriptor exceeds the metadata ring");
  float* scratch = nullptr;
  CS_HIP(cs::static_decode_scratch(&scratch), "hipGetSymbolAddress(decode scratch)");
  if ((st = use_stream(p, as_stream(stream))) != CS_OK) return st;
  DecodeWork w;
  if ((st = upload2(p, plan.convs, plan.order, &w.convs, &w.order)) != CS_OK) return st;
  const cs::PoolGeom g = p->geom();
  // untimed launches: the timing events of cs_profile_* would be created on demand
  CS_HIP(cs::launch_decode_split(g, layer, w.convs, w.order, static_cast<int>(plan.convs.size()), plan.n_items,
                                 plan.split_tokens, q, scratch, plan.single_item ? out : nullptr, p->stream),
         "decode split launch");
  if (plan.single_item) return CS_OK;
  CS_HIP(cs::launch_decode_merge(g, w.convs, static_cast<int>(plan.convs.size()), scratch, out, p->stream),
         "decode merge launch");
  return CS_OK;
}

cs_status cs_kv_pack_size(const cs_pool* p, cs_conv conv, size_t* bytes) {
  if (!p || !bytes) return fail(CS_EINVAL, "null argument");
  const cs::Conv* c = p->convs.find(conv);
  if (!c) return fail(CS_ENOENT, "unknown conversation handle");
  *bytes = wire_size(p->desc, c->len);
  return CS_OK;
}

cs_status cs_kv_pack(const cs_pool* pc, cs_conv conv, void* dst, size_t dst_bytes, cs_stream stream) {
  cs_pool* p = const_cast<cs_pool*>(pc);  // host metadata is unchanged; stream/ring state is not
  if (!p) return fail(CS_EINVAL, "null pool");
  const cs::Conv* c = p->convs.find(conv);
  if (!c) return fail(CS_ENOENT, "unknown conversation handle");
  if (dst_bytes != wire_size(p->desc, c->len)) return fail(CS_EINVAL, "dst_bytes != cs_kv_pack_size");
  if (c->len == 0) return CS_OK;
  if (!dst) return fail(CS_EINVAL, "null dst");
  cs_status st;
  if ((st = ensure_device(p)) != CS_OK) return st;
  if ((st = use_stream(p, as_stream(stream))) != CS_OK) return st;
  return timed_launch(p, CS_PROF_PACK, "pack launch", [&] {
    return cs::launch_pack(p->geom(), cs::ConvTable::slot_of(conv), c->len, dst, p->stream);
  });
}

cs_status cs_kv_unpack(cs_pool* p, const void* src, size_t src_bytes, int64_t n_tokens,
                       cs_conv* out_conv, cs_stream stream) {
  if (!p || !out_conv) return fail(CS_EINVAL, "null argument");
  if (n_tokens < 1) return fail(CS_EINVAL, "n_tokens must be >= 1");
  if (!src) return fail(CS_EINVAL, "null src");
  const int64_t np = cs::pages_for(n_tokens);
  if (np > p->desc.max_pages_per_conv) return fail(CS_ERANGE, "conversation exceeds max_pages_per_conv");
  if (src_bytes != wire_size(p->desc, n_tokens))
    return fail(CS_EINVAL, "src_bytes does not match the wire size of n_tokens for this pool");
  if (p->convs.live_count() >= p->convs.max_convs()) return fail(CS_ENOMEM, "all conversation slots are live");
  if (np > p->pages.free_count()) return fail(CS_ENOMEM, "KV pool exhausted");
  cs_status st;
  if ((st = ensure_device(p)) != CS_OK) return st;
  if ((st = use_stream(p, as_stream(stream))) != CS_OK) return st;
  cs_conv h;
  p->convs.create(&h);
  cs::Conv* c = p->convs.find(h);
  p->pages.alloc(np, c->pages);
  c->len = n_tokens;
  *out_conv = h;
  const size_t per = kQuarter / sizeof(int32_t) - 64;
  for (size_t p0 = 0; p0 < c->pages.size(); p0 += per) {
    const size_t p1 = std::min(c->pages.size(), p0 + per);
    void* d = nullptr;
    if ((st = upload(p, c->pages.data() + p0, (p1 - p0) * sizeof(int32_t), &d)) != CS_OK) return st;
    st = timed_launch(p, CS_PROF_UNPACK, "unpack launch", [&] {
      return cs::launch_unpack(p->geom(), src, static_cast<const int32_t*>(d), cs::ConvTable::slot_of(h),
                               n_tokens, static_cast<int>(p0), static_cast<int>(p1 - p0), p->stream);
    });
    if (st != CS_OK) return st;
  }
  return CS_OK;
}

cs_status cs_mixed_step(cs_pool* p, int32_t n_ext, const cs_conv* ext_convs, const int32_t* ext_lens,
                        int32_t n_dec, const cs_conv* dec_convs, const void* k, const void* v,
                        const void* q_ext, void* out_ext, const void* q_dec, void* out_dec,
                        uint32_t flags, cs_stream stream) {
  if (!p) return fail(CS_EINVAL, "null pool");
  if (n_ext < 0 || n_dec < 0) return fail(CS_EINVAL, "negative batch size");
  if (flags & ~static_cast<uint32_t>(CS_MIXED_LAYER_ORDERED)) return fail(CS_EINVAL, "unknown flags");
  if ((n_ext > 0 && (!ext_convs || !ext_lens)) || (n_dec > 0 && !dec_convs))
    return fail(CS_EINVAL, "null conversation or length array");
  std::vector<cs_conv> all;
  if (n_ext > 0) all.assign(ext_convs, ext_convs + n_ext);
  if (n_dec > 0) all.insert(all.end(), dec_convs, dec_convs + n_dec);
  std::vector<const cs::Conv*> cv;
  cs_status st = check_convs(p, static_cast<int32_t>(all.size()), all.data(), cv);
  if (st != CS_OK) return st;
  std::vector<int32_t> n_new;
  int64_t ext_rows = 0;
  for (int32_t i = 0; i < n_ext; ++i) {
    if (ext_lens[i] < 1) return fail(CS_EINVAL, "an extend chunk must hold at least one token");
    ext_rows += ext_lens[i];
    n_new.push_back(ext_lens[i]);
  }
  if (ext_rows > INT32_MAX) return fail(CS_EINVAL, "too many extend tokens");
  n_new.insert(n_new.end(), static_cast<size_t>(n_dec), 1);
  if (all.empty()) return CS_OK;
  if ((ext_rows > 0 && (!q_ext || !out_ext)) || (n_dec > 0 && (!q_dec || !out_dec)))
    return fail(CS_EINVAL, "null q/out");
  if (align_up(static_cast<size_t>(n_ext) * sizeof(cs::ExtendConvDesc), 16) + kAlign +
          sizeof(cs::ExtendTile) > kQuarter)
    return fail(CS_ENOMEM, "batch descriptor exceeds the metadata ring");
  // The decode plan covers each decoding conversation with its new token; it is checked before
  // the append so that a batch it cannot take leaves the pool unchanged.
  std::vector<int32_t> d_slots(n_dec);
  std::vector<int64_t> d_lens(n_dec);
  for (int32_t i = 0; i < n_dec; ++i) {
    d_slots[i] = cs::ConvTable::slot_of(dec_convs[i]);
    d_lens[i] = cv[n_ext + i]->len + 1;
  }
  cs::DecodePlan d_plan;
  if (n_dec > 0) {
    d_plan = plan_decode_batch(p, d_slots, d_lens);
    if ((st = check_decode_plan(p, d_plan)) != CS_OK) return st;
  }
  // append every new token (all layers); validates capacity and commits the host metadata
  if ((st = append_impl(p, static_cast<int32_t>(all.size()), all.data(), n_new.data(), k, v, stream)) != CS_OK)
    return st;
  std::vector<int32_t> e_slots(n_ext), e_q(n_new.begin(), n_new.begin() + n_ext);
  std::vector<int64_t> e_lens(n_ext);
  for (int32_t i = 0; i < n_ext; ++i) {
    e_slots[i] = cs::ConvTable::slot_of(ext_convs[i]);
    e_lens[i] = p->convs.find(ext_convs[i])->len;
  }
  ExtendWork ew;
  DecodeWork dw;
  if (n_ext > 0 && (st = upload_extend(p, e_slots, e_lens, e_q, &ew)) != CS_OK) return st;
  if (n_dec > 0 && (st = upload_decode(p, d_plan, &dw)) != CS_OK) return st;
  const size_t row_bytes = static_cast<size_t>(p->desc.n_q_heads) * p->desc.head_dim * 2;
  const int nl = p->desc.n_layers;
  const size_t ext_layer_bytes = static_cast<size_t>(ext_rows) * row_bytes;
  const size_t dec_layer_bytes = static_cast<size_t>(n_dec) * row_bytes;
  auto q_e = [&](int l) { return static_cast<const char*>(q_ext) + l * ext_layer_bytes; };
  auto o_e = [&](int l) { return static_cast<char*>(out_ext) + l * ext_layer_bytes; };
  auto q_d = [&](int l) { return static_cast<const char*>(q_dec) + l * dec_layer_bytes; };
  auto o_d = [&](int l) { return static_cast<char*>(out_dec) + l * dec_layer_bytes; };
  // Extend chunks and decode tokens are independent once their K/V is appended: with both present
  // the extend launches go to a second stream (forked from `stream`, joined back before the call
  // returns), so the matrix-core-bound extend work overlaps the HBM-bound decode work.
  const bool fork = n_ext > 0 && n_dec > 0;
  // layer order with one launch per layer (extend tiles + decode split) needs no second stream
  const bool fused_layers = (flags & CS_MIXED_LAYER_ORDERED) && fork && p->desc.head_dim == 128 &&
                            ew.parts.size() == 1;
  hipStream_t ext_stream = p->stream;
  if (fork && !fused_layers && (st = ensure_side(p)) != CS_OK) return st;
  if (fork && !fused_layers) ext_stream = p->side;
  auto fork_side = [&]() -> cs_status {
    CS_HIP(hipEventRecord(p->fork_ev, p->stream), "hipEventRecord");
    CS_HIP(hipStreamWaitEvent(p->side, p->fork_ev, 0), "hipStreamWaitEvent");
    return CS_OK;
  };
  auto join_side = [&]() -> cs_status {
    CS_HIP(hipEventRecord(p->join_ev, p->side), "hipEventRecord");
    CS_HIP(hipStreamWaitEvent(p->stream, p->join_ev, 0), "hipStreamWaitEvent");
    return CS_OK;
  };
  if (fused_layers) {
    // As in a model forward pass, one layer after the other; each layer is one launch with its
    // extend tiles and its decode split, then the decode merge.
    const cs::PoolGeom g = p->geom();
    const auto& pw = ew.parts[0];
    for (int layer = 0; layer < nl && st == CS_OK; ++layer) {
      st = timed_launch(p, CS_PROF_MIXED_LAYER, "mixed layer launch", [&] {
        return cs::launch_mixed_layer(g, layer, pw.convs, pw.tiles, pw.n_tiles, q_e(layer), o_e(layer),
                                      dw.convs, dw.order, dw.n_convs, dw.n_items, dw.split, q_d(layer),
                                      p->partials(), dw.single ? o_d(layer) : nullptr, p->stream);
      });
      if (st == CS_OK && !dw.single)
        st = timed_launch(p, CS_PROF_DECODE_MERGE, "decode merge launch", [&] {
          return cs::launch_decode_merge(g, dw.convs, dw.n_convs, p->partials(), o_d(layer), p->stream);
        });
    }
    return st;
  }
  if (flags & CS_MIXED_LAYER_ORDERED) {
    // As in a model forward pass: layer l's extend and decode overlap each other, and layer l+1
    // starts only once both are complete.
    for (int layer = 0; layer < nl && st == CS_OK; ++layer) {
      if (fork && (st = fork_side()) != CS_OK) return st;
      if (n_ext > 0) st = launch_extend_layer(p, ew, layer, q_e(layer), o_e(layer), ext_stream);
      if (n_dec > 0 && st == CS_OK) st = launch_decode_layer(p, dw, layer, q_d(layer), o_d(layer));
      if (fork) {  // join even after a failed launch, so later work never overtakes the side stream
        const cs_status sj = join_side();
        if (st == CS_OK) st = sj;
      }
    }
    return st;
  }
  // Every layer's queries are inputs of this call, so no layer waits for another: the extend
  // launches of all layers run on the side stream while the main stream decodes all layers.
  if (fork && (st = fork_side()) != CS_OK) return st;
  if (n_ext > 0) st = span_begin(p, ext_stream, CS_PROF_ATTN_FWD);
  for (int layer = 0; layer < nl && n_ext > 0 && st == CS_OK; ++layer)
    st = launch_extend_layer(p, ew, layer, q_e(layer), o_e(layer), ext_stream);
  if (const cs_status se = span_end(p); st == CS_OK) st = se;
  // Decode of all layers, one launch per layer: with one work item per conversation each layer's
  // split writes its output; otherwise split(0), then for l >= 1 a launch that merges layer l-1
  // and splits layer l into the other partial buffer, and finally merge(last).
  if (n_dec > 0 && st == CS_OK && dw.single) {
    const cs::PoolGeom g = p->geom();
    st = span_begin(p, p->stream, CS_PROF_DECODE_SPLIT);
    for (int layer = 0; layer < nl && st == CS_OK; ++layer)
      st = timed_launch(p, CS_PROF_DECODE_SPLIT, "decode split launch", [&] {
        return cs::launch_decode_split(g, layer, dw.convs, dw.order, dw.n_convs, dw.n_items, dw.split, q_d(layer),
                                       p->partials(), o_d(layer), p->stream);
      });
    if (const cs_status se = span_end(p); st == CS_OK) st = se;
  } else if (n_dec > 0 && st == CS_OK) {
    const cs::PoolGeom g = p->geom();
    float* buf[2] = {p->partials(), p->partials2()};
    st = span_begin(p, p->stream, CS_PROF_DECODE_SPLIT);
    if (st == CS_OK) st = timed_launch(p, CS_PROF_DECODE_SPLIT, "decode split launch", [&] {
      return cs::launch_decode_split(g, 0, dw.convs, dw.order, dw.n_convs, dw.n_items, dw.split, q_d(0), buf[0],
                                     nullptr, p->stream);
    });
    for (int layer = 1; layer < nl && st == CS_OK; ++layer) {
      st = timed_launch(p, CS_PROF_DECODE_SPLIT, "decode merge+split launch", [&] {
        return cs::launch_decode_merge_split(g, layer, dw.convs, dw.order, dw.n_convs, dw.n_items, dw.split,
                                             q_d(layer), buf[layer % 2], buf[(layer - 1) % 2],
                                             o_d(layer - 1), p->stream);
      });
    }
    if (const cs_status se = span_end(p); st == CS_OK) st = se;
    if (st == CS_OK)
      st = timed_launch(p, CS_PROF_DECODE_MERGE, "decode merge launch", [&] {
        return cs::launch_decode_merge(g, dw.convs, dw.n_convs, buf[(nl - 1) % 2], o_d(nl - 1),
                                       p->stream);
      });
  }
  if (fork) {  // join even after a failed launch, so later work never overtakes the side stream
    const cs_status sj = join_side();
    if (st == CS_OK) st = sj;
  }
  return st;
}

cs_status cs_device_info(int32_t device, cs_device_info_t* out) {
  if (!out) return fail(CS_EINVAL, "null out");
  hipDeviceProp_t pr;
  CS_HIP(hipGetDeviceProperties(&pr, device), "hipGetDeviceProperties");
  std::memset(out, 0, sizeof(*out));
  std::strncpy(out->name, pr.name, sizeof(out->name) - 1);
  std::strncpy(out->arch, pr.gcnArchName, sizeof(out->arch) - 1);
  out->cu_count = pr.multiProcessorCount;
  out->clock_khz = pr.clockRate;
  out->memory_clock_khz = pr.memoryClockRate;
  out->memory_bus_width_bits = pr.memoryBusWidth;
  out->lds_per_cu_bytes = static_cast<int64_t>(pr.maxSharedMemoryPerMultiProcessor);
  out->lds_per_block_bytes = static_cast<int64_t>(pr.sharedMemPerBlock);
  out->l2_bytes = pr.l2CacheSize;
  out->total_mem_bytes = static_cast<int64_t>(pr.totalGlobalMem);
  return CS_OK;
}

cs_status cs_probe_stream_read(const void* src, size_t bytes, void* sink, cs_stream stream) {
  if (!src || !sink) return fail(CS_EINVAL, "null src or sink");
  if (bytes % 16) return fail(CS_EINVAL, "bytes must be a multiple of 16");
  int dev = 0, cus = 0;
  CS_HIP(hipGetDevice(&dev), "hipGetDevice");
  CS_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev), "hipDeviceGetAttribute");
  CS_HIP(cs::launch_stream_read_probe(src, bytes, static_cast<uint32_t*>(sink), cus, as_stream(stream)),
         "stream read probe launch");
  return CS_OK;
}

cs_status cs_debug_fail_launches(cs_pool* p, int64_t after) {
  if (!p) return fail(CS_EINVAL, "null pool");
  p->fail_after = after < 0 ? -1 : after;
  return CS_OK;
}

cs_status cs_profile_start(cs_pool* p) {
  if (!p) return fail(CS_EINVAL, "null pool");
  for (auto& pe : p->prof_events) {
    p->ev_free.push_back(pe.start);
    p->ev_free.push_back(pe.stop);
  }
  p->prof_events.clear();
  p->prof_on = true;
  return CS_OK;
}

cs_status cs_profile_stop(cs_pool* p, double* ms, int64_t* launches) {
  if (!p || !ms || !launches) return fail(CS_EINVAL, "null argument");
  for (int k = 0; k < CS_PROF_KINDS; ++k) {
    ms[k] = 0.0;
    launches[k] = 0;
  }
  p->prof_on = false;
  for (auto& pe : p->prof_events) {
    CS_HIP(hipEventSynchronize(pe.stop), "hipEventSynchronize");
    float t = 0.f;
    CS_HIP(hipEventElapsedTime(&t, pe.start, pe.stop), "hipEventElapsedTime");
    ms[pe.kind] += t;
    launches[pe.kind] += pe.launches;
    p->ev_free.push_back(pe.start);
    p->ev_free.push_back(pe.stop);
  }
  p->prof_events.clear();
  return CS_OK;
}

}  // extern "C"
namespace cs {
// Error reporting shared with the other C-ABI translation units (sched_capi.cpp).
cs_status api_fail(cs_status code, const char* msg) { return fail(code, msg); }
}  // namespace cs
