#include "host_state.hpp"

#include <algorithm>
#include <numeric>

namespace cs {

PagePool::PagePool(int64_t n_pages, uint64_t seed) : n_pages_(n_pages), rng_(seed) {
  free_.resize(static_cast<size_t>(n_pages));
  std::iota(free_.begin(), free_.end(), 0);
  // Fisher-Yates shuffle: physical placement of logical pages is random.
  for (int64_t i = n_pages - 1; i > 0; --i) {
    int64_t j = static_cast<int64_t>(rng_.below(static_cast<uint64_t>(i + 1)));
    std::swap(free_[i], free_[j]);
  }
}

bool PagePool::alloc(int64_t n, std::vector<int32_t>& out) {
  if (n < 0 || n > free_count()) return false;
  out.reserve(out.size() + static_cast<size_t>(n));
  for (int64_t i = 0; i < n; ++i) {
    out.push_back(free_.back());
    free_.pop_back();
  }
  return true;
}

void PagePool::release(const std::vector<int32_t>& pages) {
  for (int32_t p : pages) {
    free_.push_back(p);
    // keep the free list in random order: swap the returned page to a random position
    size_t j = static_cast<size_t>(rng_.below(free_.size()));
    std::swap(free_[j], free_.back());
  }
}

void PagePool::unalloc(const std::vector<int32_t>& pages) {
  for (auto it = pages.rbegin(); it != pages.rend(); ++it) free_.push_back(*it);
}

ConvTable::ConvTable(int32_t max_convs, int32_t max_pages_per_conv)
    : max_convs_(max_convs), max_pages_(max_pages_per_conv), slots_(static_cast<size_t>(max_convs)) {
  for (int32_t i = 0; i < max_convs; ++i) free_slots_.push_back(i);
}

bool ConvTable::create(int32_t* handle) {
  if (free_slots_.empty()) return false;
  int32_t s = free_slots_.front();
  free_slots_.pop_front();
  Conv& c = slots_[static_cast<size_t>(s)];
  c.live = true;
  c.len = 0;
  c.pages.clear();
  ++live_;
  *handle = s | static_cast<int32_t>((c.gen & 0x7FFu) << kSlotBits);
  return true;
}

Conv* ConvTable::find(int32_t handle) {
  if (handle < 0) return nullptr;
  int32_t s = slot_of(handle);
  if (s >= max_convs_) return nullptr;
  Conv& c = slots_[static_cast<size_t>(s)];
  if (!c.live) return nullptr;
  if (static_cast<uint32_t>(handle >> kSlotBits) != (c.gen & 0x7FFu)) return nullptr;
  return &c;
}

const Conv* ConvTable::find(int32_t handle) const {
  return const_cast<ConvTable*>(this)->find(handle);
}

void ConvTable::destroy(int32_t handle, PagePool& pool) {
  int32_t s = slot_of(handle);
  Conv& c = slots_[static_cast<size_t>(s)];
  pool.release(c.pages);
  c.pages.clear();
  c.pages.shrink_to_fit();
  c.len = 0;
  c.live = false;
  c.gen = (c.gen + 1) & 0x7FFu;
  --live_;
  free_slots_.push_back(s);
}

DecodePlan plan_decode(const std::vector<int32_t>& slots, const std::vector<int64_t>& lens,
                       int32_t n_kv_heads, int64_t target_items) {
  static const int32_t kCandidates[] = {1024, 512, 256, 128};
  DecodePlan plan;
  for (int32_t split : kCandidates) {
    int64_t items = 0;
    for (int64_t L : lens) items += (L + split - 1) / split;
    plan.split_tokens = split;
    if (items * n_kv_heads >= target_items) break;
  }
  const int32_t split = plan.split_tokens;
  const int64_t item_keys = static_cast<int64_t>(kDecodeSubSplits) * split;
  int32_t start = 0;
  plan.convs.reserve(lens.size());
  for (size_t i = 0; i < lens.size(); ++i) {
    int32_t ns = static_cast<int32_t>((lens[i] + item_keys - 1) / item_keys);
    plan.convs.push_back({slots[i], static_cast<int32_t>(lens[i]), start, ns});
    start += ns;
  }
  plan.n_items = start;
  plan.single_item = start == static_cast<int32_t>(lens.size());
  std::vector<int64_t> keys(static_cast<size_t>(start));
  for (const DecodeConvDesc& c : plan.convs)
    for (int32_t s = 0; s < c.n_splits; ++s) keys[c.item_start + s] = std::min<int64_t>(item_keys, c.len - s * item_keys);
  plan.order.resize(static_cast<size_t>(start));
  std::iota(plan.order.begin(), plan.order.end(), 0);
  std::stable_sort(plan.order.begin(), plan.order.end(),
                   [&](int32_t x, int32_t y) { return keys[x] > keys[y]; });
  return plan;
}

ExtendPlan plan_extend(const std::vector<int32_t>& slots, const std::vector<int64_t>& lens,
                       const std::vector<int32_t>& q_lens, int32_t q_tile) {
  ExtendPlan plan;
  plan.q_tile = q_tile;
  int32_t row = 0;
  std::vector<std::pair<int64_t, ExtendTile>> work;
  for (size_t i = 0; i < lens.size(); ++i) {
    plan.convs.push_back({slots[i], static_cast<int32_t>(lens[i]), q_lens[i], row});
    row += q_lens[i];
    for (int32_t q0 = 0; q0 < q_lens[i]; q0 += q_tile) {
      int64_t keys = lens[i] - q_lens[i] + std::min(q_lens[i], q0 + q_tile);
      work.push_back({keys, {static_cast<int32_t>(i), q0}});
    }
  }
  // Conversation-major order: longest conversation first, its heaviest tiles first. Workgroups that
  // run at the same time on one XCD then mostly belong to one conversation and sweep the same
  // prefix K/V, so it stays in that XCD's L2; the heaviest tiles still start first.
  std::vector<int64_t> conv_keys(lens.size(), 0);
  for (auto& w : work) conv_keys[w.second.conv] = std::max(conv_keys[w.second.conv], w.first);
  std::stable_sort(work.begin(), work.end(), [&](const auto& a, const auto& b) {
    const int64_t ka = conv_keys[a.second.conv], kb = conv_keys[b.second.conv];
    if (ka != kb) return ka > kb;
    if (a.second.conv != b.second.conv) return a.second.conv < b.second.conv;
    return a.first > b.first;
  });
  plan.tiles.reserve(work.size());
  for (auto& w : work) plan.tiles.push_back(w.second);
  return plan;
}

std::vector<PageChunk> plan_append(const std::vector<int32_t>& slots,
                                   const std::vector<int64_t>& lens,
                                   const std::vector<int32_t>& n_new,
                                   const std::vector<const std::vector<int32_t>*>& page_lists) {
  std::vector<PageChunk> chunks;
  int64_t row_base = 0;
  for (size_t i = 0; i < lens.size(); ++i) {
    const int64_t pos0 = lens[i], n = n_new[i];
    if (n > 0) {
      const int64_t old_pages = pages_for(pos0);
      for (int64_t p = pos0 / kPage; p <= (pos0 + n - 1) / kPage; ++p) {
        const int64_t a = std::max(pos0, p * kPage), b = std::min(pos0 + n, (p + 1) * kPage);
        PageChunk c;
        c.conv = static_cast<int32_t>(i);
        c.slot = slots[i];
        c.lpage = static_cast<int32_t>(p);
        c.page = (*page_lists[i])[static_cast<size_t>(p)];
        c.t0 = static_cast<int32_t>(a - p * kPage);
        c.t1 = static_cast<int32_t>(b - p * kPage);
        c.src_row = static_cast<int32_t>(row_base + (a - pos0));
        c.new_page = p >= old_pages ? 1 : 0;
        chunks.push_back(c);
      }
    }
    row_base += n;
  }
  return chunks;
}

}  // namespace cs
