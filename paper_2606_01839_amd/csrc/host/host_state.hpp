// Host-side metadata of a KV page pool: free-page list with seeded random placement, the
// conversation table (length + logical->physical page list per conversation), and the work plans
// the attention kernels are launched with. No HIP here: everything compiles and is tested on a CPU.
#pragma once

#include <cstdint>
#include <deque>
#include <string>
#include <vector>

namespace cs {

constexpr int kPage = 16;  // tokens per KV page

inline int64_t pages_for(int64_t tokens) { return (tokens + kPage - 1) / kPage; }

// SplitMix64 (Steele, Lea, Flood 2014) -- seeds the page-placement shuffle.
struct SplitMix64 {
  uint64_t s;
  explicit SplitMix64(uint64_t seed) : s(seed) {}
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  uint64_t below(uint64_t n) { return next() % n; }  // modulo bias is irrelevant for placement
};

// Fixed set of physical pages handed out in a seeded random order.
class PagePool {
 public:
  PagePool(int64_t n_pages, uint64_t seed);
  int64_t capacity() const { return n_pages_; }
  int64_t free_count() const { return static_cast<int64_t>(free_.size()); }
  int64_t used_count() const { return n_pages_ - free_count(); }
  // All-or-nothing: appends n page ids to `out` and returns true, or changes nothing.
  bool alloc(int64_t n, std::vector<int32_t>& out);
  void release(const std::vector<int32_t>& pages);
  // Undo the latest alloc calls exactly: `pages` are the ids they handed out, in order (the free
  // list then holds the same ids in the same order as before them).
  void unalloc(const std::vector<int32_t>& pages);

 private:
  int64_t n_pages_;
  std::vector<int32_t> free_;
  SplitMix64 rng_;
};

struct Conv {
  bool live = false;
  uint32_t gen = 0;
  int64_t len = 0;
  std::vector<int32_t> pages;  // logical page i -> physical page id
};

// Conversation handles are slot | (generation << 20): a destroyed handle stays invalid after its
// slot is reused (until the 11-bit generation wraps). Freed slots are reused first-in first-out.
class ConvTable {
 public:
  static constexpr int kSlotBits = 20;
  ConvTable(int32_t max_convs, int32_t max_pages_per_conv);
  int32_t max_convs() const { return max_convs_; }
  int32_t max_pages_per_conv() const { return max_pages_; }
  int32_t live_count() const { return live_; }
  bool create(int32_t* handle);               // false when every slot is live
  Conv* find(int32_t handle);                  // nullptr if unknown / destroyed
  const Conv* find(int32_t handle) const;
  static int32_t slot_of(int32_t handle) { return handle & ((1 << kSlotBits) - 1); }
  void destroy(int32_t handle, PagePool& pool);  // handle must be valid

 private:
  int32_t max_convs_, max_pages_, live_ = 0;
  std::vector<Conv> slots_;
  std::deque<int32_t> free_slots_;
};

// ---------------------------------------------------------------------------------------------
// Work plans (plain structs uploaded to the device as-is; layouts shared with the kernels).
// ---------------------------------------------------------------------------------------------

// Decode: one work item = (conversation b, item s, kv head) covers keys [s*K, min(len, (s+1)*K))
// with K = kDecodeSubSplits * split_tokens, shared out evenly over its waves in whole page pairs.
// Items of conversation b are numbered item_start[b] + s.
struct DecodeConvDesc {
  int32_t slot;        // row of the device page-table mirror
  int32_t len;         // tokens
  int32_t item_start;  // first work item of this conversation
  int32_t n_splits;    // work items: ceil(len / (kDecodeSubSplits * split_tokens))
};

// Waves per decode work item: each takes one split of keys; the item's waves merge their partial
// results on chip and write one partial record per query head.
constexpr int kDecodeSubSplits = 8;

struct DecodePlan {
  int32_t split_tokens = 0;  // keys per wave (one split), multiple of 32, <= 1024
  int32_t n_items = 0;       // work items over the batch (per kv head)
  bool single_item = false;  // every conversation is one work item (no merge of items needed)
  std::vector<DecodeConvDesc> convs;
  // Launch order: workgroup w takes item order[w / n_kv_heads]. Full items (K keys) come first, in
  // conversation order, then the shorter last items by decreasing key count, so the last round
  // of workgroups on the chip holds the shortest ones.
  std::vector<int32_t> order;
};

// Choose the split size: the largest candidate for which the splits holding keys, over all kv
// heads, number at least `target_items` (the waves that read), else the smallest candidate. A
// work item is kDecodeSubSplits consecutive splits of one conversation.
DecodePlan plan_decode(const std::vector<int32_t>& slots, const std::vector<int64_t>& lens,
                       int32_t n_kv_heads, int64_t target_items);

// Extend / prefill: queries are the last q_len tokens of each conversation, tiled by 64 query
// tokens; one tile = (conversation, 64-token query block) x one kv head.
struct ExtendConvDesc {
  int32_t slot;
  int32_t len;    // tokens (keys) of the conversation
  int32_t q_len;  // queries = positions len-q_len .. len-1
  int32_t q_row;  // first row of this conversation in the q/out tensors
};

struct ExtendTile {
  int32_t conv;   // index into the batch
  int32_t q0;     // first query index (0-based within the conversation's q_len)
};

struct ExtendPlan {
  int32_t q_tile = 64;
  std::vector<ExtendConvDesc> convs;
  std::vector<ExtendTile> tiles;  // conversation-major (longest conversation first), heaviest tile first
};

ExtendPlan plan_extend(const std::vector<int32_t>& slots, const std::vector<int64_t>& lens,
                       const std::vector<int32_t>& q_lens, int32_t q_tile);

// Append / unpack: one chunk = the part of one logical page a call writes.
struct PageChunk {
  int32_t conv;      // index into the batch
  int32_t slot;      // page-table row
  int32_t lpage;     // logical page index within the conversation
  int32_t page;      // physical page id
  int32_t t0, t1;    // token slots [t0, t1) of the page receive data; when t0 = 0, [t1, 16) are zeroed
  int32_t src_row;   // row (token) of the first written slot in the source tensor
  int32_t new_page;  // 1 if this page was just allocated (the mirror entry must be written)
};

// Chunks for appending n_new[i] tokens to conversations whose lengths are lens[i] and whose page
// lists already include the newly reserved pages.
std::vector<PageChunk> plan_append(const std::vector<int32_t>& slots,
                                   const std::vector<int64_t>& lens,
                                   const std::vector<int32_t>& n_new,
                                   const std::vector<const std::vector<int32_t>*>& page_lists);

}  // namespace cs
