// Host-metadata unit test (page pool, conversation table, plans); built with -fsanitize=address,
// undefined by tests/test_host_cpp.py. Exits non-zero on the first failed check.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <set>
#include <vector>

#include "host/host_state.hpp"
#include "host/sched.hpp"

#define CHECK(c)                                                          \
  do {                                                                    \
    if (!(c)) {                                                           \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
      std::exit(1);                                                       \
    }                                                                     \
  } while (0)

static void pool_basics() {
  cs::PagePool a(100, 7), b(100, 7), c(100, 8);
  std::vector<int32_t> pa, pb, pc;
  CHECK(a.alloc(100, pa) && b.alloc(100, pb) && c.alloc(100, pc));
  CHECK(pa == pb);                 // same seed, same placement
  CHECK(pa != pc);                 // another seed, another placement
  std::vector<int32_t> sorted = pa;
  std::sort(sorted.begin(), sorted.end());
  for (int i = 0; i < 100; ++i) CHECK(sorted[i] == i);  // a permutation of all pages
  CHECK(a.free_count() == 0 && a.used_count() == 100);
  std::vector<int32_t> more;
  CHECK(!a.alloc(1, more) && more.empty());             // all-or-nothing
  a.release(std::vector<int32_t>(pa.begin(), pa.begin() + 10));
  CHECK(a.free_count() == 10);
  CHECK(!a.alloc(11, more) && more.empty());
  CHECK(a.alloc(10, more) && more.size() == 10);
  // unalloc undoes allocations exactly: the next allocations hand out the same ids again
  cs::PagePool u(50, 3), w(50, 3);
  std::vector<int32_t> u1, u2, w1;
  CHECK(u.alloc(7, u1) && u.alloc(5, u1));
  u.unalloc(u1);
  CHECK(u.free_count() == 50 && u.alloc(20, u2) && w.alloc(20, w1) && u2 == w1);
}

static void conv_table() {
  cs::PagePool pool(64, 1);
  cs::ConvTable t(3, 8);
  int32_t h[4];
  CHECK(t.create(&h[0]) && t.create(&h[1]) && t.create(&h[2]));
  CHECK(!t.create(&h[3]));
  CHECK(t.find(h[1]) && t.live_count() == 3);
  t.find(h[1])->len = 40;
  CHECK(pool.alloc(3, t.find(h[1])->pages));
  CHECK(pool.used_count() == 3);
  t.destroy(h[1], pool);
  CHECK(pool.used_count() == 0 && !t.find(h[1]) && t.live_count() == 2);
  CHECK(t.create(&h[3]) && h[3] != h[1] && !t.find(h[1]));  // stale handle stays invalid
  CHECK(cs::ConvTable::slot_of(h[3]) == cs::ConvTable::slot_of(h[1]));
  CHECK(!t.find(-1) && !t.find(1 << 19));
}

static void decode_plan() {
  std::vector<int32_t> slots = {4, 9, 2};
  std::vector<int64_t> lens = {1, 1000, 4096};
  cs::DecodePlan p = cs::plan_decode(slots, lens, 8, 1 << 30);  // unreachable target -> smallest split
  CHECK(p.split_tokens == 128);
  // work items of kDecodeSubSplits splits of 128 keys each
  const int64_t ik = static_cast<int64_t>(cs::kDecodeSubSplits) * 128;
  const int32_t n1 = static_cast<int32_t>((1000 + ik - 1) / ik), n2 = static_cast<int32_t>((4096 + ik - 1) / ik);
  CHECK(p.convs.size() == 3 && p.convs[0].n_splits == 1 && p.convs[1].n_splits == n1 && p.convs[2].n_splits == n2);
  CHECK(p.convs[1].item_start == 1 && p.convs[2].item_start == 1 + n1 && p.n_items == 1 + n1 + n2);
  // launch order: the full items (conversation 2's four) first, then 1000 keys, then 1 key
  CHECK(n1 == 1 && n2 == 4 && (p.order == std::vector<int32_t>{2, 3, 4, 5, 1, 0}));
  cs::DecodePlan q = cs::plan_decode(slots, lens, 8, 1);  // any split satisfies -> largest
  CHECK(q.split_tokens == 1024 && q.n_items == 3);         // one item each (4096 <= 4 * 1024)
  // the target counts splits holding keys: 1 + 1 + 4 = 6 splits of 1024 keys, x 8 kv heads = 48
  CHECK(cs::plan_decode(slots, lens, 8, 48).split_tokens == 1024);
  CHECK(cs::plan_decode(slots, lens, 8, 49).split_tokens == 512);
}

// Random batches: the items of a conversation tile [0, len) in splits of split_tokens, 8 per item;
// item_start is the prefix sum; the split is the largest candidate meeting the target (or 128);
// single_item holds exactly when every conversation is one item; the launch order is a
// permutation of the items: every full item, in item order, then the others by decreasing key
// count (ties in item order).
static void decode_plan_random() {
  std::srand(12345);
  const int32_t cands[] = {1024, 512, 256, 128};
  for (int trial = 0; trial < 200; ++trial) {
    const int n = 1 + std::rand() % 40, hkv = 1 + std::rand() % 8;
    const int64_t target = 1 + std::rand() % 8000;
    std::vector<int32_t> slots(n);
    std::vector<int64_t> lens(n);
    for (int i = 0; i < n; ++i) {
      slots[i] = i;
      lens[i] = 1 + std::rand() % (std::rand() % 2 ? 600 : 40000);
    }
    const cs::DecodePlan p = cs::plan_decode(slots, lens, hkv, target);
    int32_t expect_split = 128;
    for (int32_t sp : cands) {
      int64_t waves = 0;
      for (int64_t L : lens) waves += (L + sp - 1) / sp;
      if (waves * hkv >= target) { expect_split = sp; break; }
    }
    CHECK(p.split_tokens == expect_split);
    const int64_t ik = static_cast<int64_t>(cs::kDecodeSubSplits) * p.split_tokens;
    int32_t start = 0;
    bool single = true;
    for (int i = 0; i < n; ++i) {
      CHECK(p.convs[i].slot == slots[i] && p.convs[i].len == lens[i] && p.convs[i].item_start == start);
      CHECK(p.convs[i].n_splits == (lens[i] + ik - 1) / ik);
      // the last item of the conversation holds keys, the one after it would not
      CHECK(static_cast<int64_t>(p.convs[i].n_splits - 1) * ik < lens[i] && p.convs[i].n_splits * ik >= lens[i]);
      single = single && p.convs[i].n_splits == 1;
      start += p.convs[i].n_splits;
    }
    CHECK(p.n_items == start && p.single_item == single);
    std::vector<int64_t> keys;
    for (int i = 0; i < n; ++i)
      for (int s = 0; s < p.convs[i].n_splits; ++s) keys.push_back(std::min<int64_t>(ik, lens[i] - s * ik));
    CHECK(p.order.size() == keys.size());
    std::vector<char> seen(keys.size(), 0);
    for (size_t j = 0; j < p.order.size(); ++j) {
      const int32_t it = p.order[j];
      CHECK(it >= 0 && it < p.n_items && !seen[it]);
      seen[it] = 1;
      if (j > 0) {
        const int32_t prev = p.order[j - 1];
        CHECK(keys[prev] >= keys[it]);
        if (keys[prev] == keys[it]) CHECK(prev < it);
      }
    }
  }
}

static void extend_plan() {
  std::vector<int32_t> slots = {0, 1};
  std::vector<int64_t> lens = {100, 300};
  std::vector<int32_t> ql = {100, 130};
  cs::ExtendPlan p = cs::plan_extend(slots, lens, ql, 64);
  CHECK(p.convs[0].q_row == 0 && p.convs[1].q_row == 100);
  CHECK(p.tiles.size() == 2 + 3);
  // longest first: conversation 1 (prefix 170) tile q0=128 sees 300 keys
  CHECK(p.tiles[0].conv == 1 && p.tiles[0].q0 == 128);
  std::set<std::pair<int, int>> seen;
  for (auto& t : p.tiles) seen.insert({t.conv, t.q0});
  CHECK(seen.size() == 5 && seen.count({0, 64}) && seen.count({1, 64}));
}

static void append_plan() {
  std::vector<int32_t> pages0 = {7, 3};        // conversation with 20 tokens (2 pages) + 1 new
  std::vector<int32_t> pages1 = {5};           // empty conversation receiving 16 tokens
  std::vector<const std::vector<int32_t>*> lists = {&pages0, &pages1};
  // conversation 0: tokens 20..49 -> page 1 slots 4..15, page 2 slots 0..15, page 3 slots 0..1
  pages0.push_back(11);
  pages0.push_back(12);
  std::vector<cs::PageChunk> ch = cs::plan_append({2, 6}, {20, 0}, {30, 16}, lists);
  CHECK(ch.size() == 3 + 1);
  CHECK(ch[0].lpage == 1 && ch[0].page == 3 && ch[0].t0 == 4 && ch[0].t1 == 16 && ch[0].src_row == 0 && !ch[0].new_page);
  CHECK(ch[1].lpage == 2 && ch[1].page == 11 && ch[1].t0 == 0 && ch[1].t1 == 16 && ch[1].src_row == 12 && ch[1].new_page);
  CHECK(ch[2].lpage == 3 && ch[2].page == 12 && ch[2].t0 == 0 && ch[2].t1 == 2 && ch[2].src_row == 28 && ch[2].new_page);
  CHECK(ch[3].conv == 1 && ch[3].lpage == 0 && ch[3].t0 == 0 && ch[3].t1 == 16 && ch[3].src_row == 30 && ch[3].new_page);
}

static void placement() {
  // binding: fraction of pages used, exact for counts near 2^62 (no overflow under UBSan)
  const int64_t big = int64_t(1) << 61;
  int64_t used[3] = {big - 1, big - 2, 5}, fr[3] = {big + 1, big + 2, 0};
  CHECK(cs::least_occupied(3, used, fr, 1) == 1);
  CHECK(cs::least_occupied(3, used, fr, big + 2) == 1);
  CHECK(cs::least_occupied(3, used, fr, big + 3) == -1);
  // curve fit: exact quadratic recovered; degenerate inputs refused
  int64_t L[4] = {1000, 2000, 4000, 8000};
  double t[4];
  for (int i = 0; i < 4; ++i) t[i] = 0.5 + 2e-4 * L[i] + 3e-8 * double(L[i]) * L[i];
  cs::PrefillCurve c;
  double r2 = 0;
  CHECK(cs::fit_prefill_curve(L, t, 4, &c, &r2));
  CHECK(std::fabs(c.c0 - 0.5) < 1e-9 && std::fabs(c.c1 - 2e-4) < 1e-12 && std::fabs(c.c2 - 3e-8) < 1e-15);
  CHECK(std::fabs(r2 - 1.0) < 1e-12);
  int64_t same[3] = {7, 7, 9};
  CHECK(!cs::fit_prefill_curve(same, t, 3, &c, &r2));
  // provisioning and admission
  cs::Provisioning p;
  CHECK(cs::provision_decoders(25000, 15000, 1000, 1000, 1e9, 1, &p) && p.n_decoders == 2);
  CHECK(!cs::provision_decoders(0, 1, 1, 1, 1, 1, &p));
  cs::PrefillCurve one;
  one.c0 = 1.0;
  cs::Admission a(one, 1.5);
  double st = 0, dn = 0;
  CHECK(a.admit(10, 0.0, &st, &dn) && st == 0.0 && dn == 1.0);
  CHECK(a.admit(10, 0.2, &st, &dn) && st == 1.0 && dn == 2.0);
  CHECK(!a.admit(10, 0.4, &st, &dn) && a.busy_until() == 2.0);
}

int main() {
  placement();
  pool_basics();
  conv_table();
  decode_plan();
  decode_plan_random();
  extend_plan();
  append_plan();
  std::puts("host metadata tests passed");
  return 0;
}
