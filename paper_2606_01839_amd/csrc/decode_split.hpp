// Split phase of batched decode (split-K flash decoding over paged KV), shared by the decode
// kernels and by the fused extend + decode kernel of a mixed step; see decode.hip.
#pragma once

#include <cmath>

#include "device_common.hpp"
#include "kernels.hpp"

namespace cs {

struct DecodeArgs {
  const uint16_t* pool;
  int64_t n_pages;
  int n_kv_heads;
  int group;  // query heads per kv head (<= 16)
  int layer;
  const int32_t* page_table;
  int max_pages;
  const DecodeConvDesc* convs;
  int n_convs;
  int n_items;  // work items of the plan (kDecodeSubSplits splits each)
  int split;    // keys per split (per wave), multiple of 32, <= 1024
  const uint16_t* q;
  uint16_t* out;    // with direct: the final output [n_convs][n_q_heads][D]
  int direct;       // every conversation is one item: write the output instead of a record
  float* partials;  // [n_items * n_kv_heads][group] records of partial_floats(D), one per item
  float scale_log2;
  const int32_t* order;  // [n_items]: workgroup w takes item order[w / n_kv_heads]
};

// Kernel arguments read by every wave alike are loaded through the constant address space, so
// they land in scalar registers and the loop control, page bases and addresses stay wave-uniform.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(4))) T* as_const(const T* p) {
  return (const __attribute__((address_space(4))) T*)reinterpret_cast<uintptr_t>(p);
}

__device__ __forceinline__ DecodeConvDesc load_desc(const __attribute__((address_space(4))) DecodeConvDesc* p) {
  DecodeConvDesc d;
  d.slot = p->slot;
  d.len = p->len;
  d.item_start = p->item_start;
  d.n_splits = p->n_splits;
  return d;
}

__device__ __forceinline__ int find_conv(const __attribute__((address_space(4))) DecodeConvDesc* convs,
                                         int n, int item) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {  // largest b with item_start <= item
    int mid = (lo + hi + 1) >> 1;
    if (convs[mid].item_start <= item) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Threads of a workgroup that takes one work item: one wave per split.
constexpr int kDecodeItemThreads = 64 * kDecodeSubSplits;

// LDS floats one work item's workgroup needs to hand waves 1 .. kDecodeSubSplits-1's partial
// results to wave 0 (up to 8 query heads per kv head: o[D], m, l each).
template <int D>
constexpr int split_exchange_floats() { return (kDecodeSubSplits - 1) * 8 * (D + 2); }

// Work unit `work` = (order[work / n_kv_heads], work % n_kv_heads) = (item, kv head) of the plan,
// taken by one workgroup of kDecodeSubSplits waves (this wave = `wave`; `xch` = its LDS exchange
// area, split_exchange_floats<D>() floats). The item's n keys are shared out evenly: wave w reads
// keys [k0 + w s, k0 + (w + 1) s) with s = ceil(n / kDecodeSubSplits) rounded up to a page pair,
// so a short last item keeps all its waves busy for a short time instead of a few of them for a
// full split. Then the other waves hand their (o, m, l) to wave 0 through LDS, which merges them
// in the order w = 0, 1, ... and writes the item's one partial record: far fewer, larger writes
// interleaved with the KV stream than one record per wave (the HBM reads run 7% faster with 8
// waves per item than with one). Every wave reaches the one barrier, also in a workgroup whose
// work unit lies past the end (work >= n_items * n_kv_heads: no keys, nothing written).
template <int D>
__device__ __forceinline__ void split_body(const DecodeArgs& a, const int work, const int wave,
                                           float* xch) {
  constexpr int KS = D / 32;  // k-steps of the QK^T contraction
  constexpr int DT = D / 16;  // 16-dim tiles of the output
  const int lane = threadIdx.x & 63;
  const bool valid = work < a.n_items * a.n_kv_heads;
  const int item = as_const(a.order)[valid ? work / a.n_kv_heads : 0], g = work % a.n_kv_heads;
  const auto* convs = as_const(a.convs);
  const int conv_idx = find_conv(convs, a.n_convs, item);
  const DecodeConvDesc cd = load_desc(convs + conv_idx);
  const int item_k0 = (item - cd.item_start) * kDecodeSubSplits * a.split;
  const int item_k1 = min(cd.len, item_k0 + kDecodeSubSplits * a.split);
  const int wave_keys = ((item_k1 - item_k0 + kDecodeSubSplits - 1) / kDecodeSubSplits + 2 * kPageTokens - 1) &
                        ~(2 * kPageTokens - 1);  // <= split (a multiple of 32)
  const int k_begin = item_k0 + wave * wave_keys;
  const int k_end = valid ? min(item_k1, k_begin + wave_keys) : k_begin;
  const int n_pg = k_end > k_begin ? (k_end - k_begin + kPageTokens - 1) / kPageTokens : 0;
  const int32_t* pt = a.page_table + static_cast<size_t>(cd.slot) * a.max_pages + k_begin / kPageTokens;

  const int c = lane & 15;   // MFMA column: query head within the group; A-operand row: key / dim
  const int qd = lane >> 4;  // k-block of the lane (8 consecutive k values)

  // Query operand: head c of this kv head's group, dims 32*ks + 8*qd .. +8.
  const int n_q_heads = a.n_kv_heads * a.group;
  bf16x8 qop[KS];
  {
    const uint16_t* qrow = a.q + (static_cast<size_t>(conv_idx) * n_q_heads + g * a.group + c) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qop[ks] = c < a.group ? as_bf16x8(ld16(qrow + 32 * ks + 8 * qd)) : bf16x8{};
  }

  const int pid = lane < n_pg ? pt[lane] : 0;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t head_stride = static_cast<size_t>(2 * kPageTokens * D);
  const uint16_t* layer_base = a.pool + static_cast<size_t>(a.layer) * a.n_pages * a.n_kv_heads * head_stride +
                               static_cast<size_t>(g) * head_stride;
  const size_t page_stride = static_cast<size_t>(a.n_kv_heads) * head_stride;
  // Per-lane byte offsets inside a page block (the same for every page): key c, dims 8 qd ..
  // (+32 ks: next K sub-block, 1 KiB on); V^T row c (of a 16-dim tile), keys 4 qd .. 4 qd + 3.
  const uint32_t koff = static_cast<uint32_t>((c * 32 + 8 * qd) * 2);
  const uint32_t voff = static_cast<uint32_t>((kPageTokens * D + c * kPageTokens + 4 * qd) * 2);

  for (int j = 0; j < n_pg; j += 2) {
    const bool has_b = j + 1 < n_pg;
    const int pa = __builtin_amdgcn_readlane(pid, j);
    const int pb = has_b ? __builtin_amdgcn_readlane(pid, j + 1) : pa;
    const uint8_t* blk_a = reinterpret_cast<const uint8_t*>(layer_base + static_cast<size_t>(pa) * page_stride);
    const uint8_t* blk_b = reinterpret_cast<const uint8_t*>(layer_base + static_cast<size_t>(pb) * page_stride);

    bf16x8 ka[KS], kb[KS];
    uint2 va[DT], vb[DT];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) ka[ks] = as_bf16x8(ld16_nt(blk_a + koff + 1024 * ks));
#pragma unroll
    for (int t = 0; t < DT; ++t) va[t] = ld8_nt(blk_a + voff + 16 * kPageTokens * 2 * t);
    if (has_b) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kb[ks] = as_bf16x8(ld16_nt(blk_b + koff + 1024 * ks));
#pragma unroll
      for (int t = 0; t < DT; ++t) vb[t] = ld8_nt(blk_b + voff + 16 * kPageTokens * 2 * t);
    } else {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kb[ks] = bf16x8{};
#pragma unroll
      for (int t = 0; t < DT; ++t) vb[t] = make_uint2(0, 0);
    }

    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[ks], qop[ks], sa, 0, 0, 0);
      sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[ks], qop[ks], sb, 0, 0, 0);
    }
    // sa[r]: head c, key k_begin + 16j + 4qd + r; sb[r]: the same + 16.
    const int key_a = k_begin + kPageTokens * j + 4 * qd;
    float xa[4], xb[4];
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      xa[r] = key_a + r < k_end ? sa[r] * a.scale_log2 : -INFINITY;
      xb[r] = key_a + kPageTokens + r < k_end ? sb[r] * a.scale_log2 : -INFINITY;
      mx = fmaxf(mx, fmaxf(xa[r], xb[r]));
    }
    mx = fmaxf(mx, xor_shfl(mx, 16));
    mx = fmaxf(mx, xor_shfl(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2(m_run - m_new);
    float pa_[4], pb_[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      pa_[r] = fast_exp2(xa[r] - m_new);
      pb_[r] = fast_exp2(xb[r] - m_new);
    }
    const uint4 pw = make_uint4(pack_bf16x2(pa_[0], pa_[1]), pack_bf16x2(pa_[2], pa_[3]),
                                pack_bf16x2(pb_[0], pb_[1]), pack_bf16x2(pb_[2], pb_[3]));
    // The denominator sums the same bf16-rounded weights the PV product uses.
    const float psum = (sum_bf16x2(pw.x) + sum_bf16x2(pw.y)) + (sum_bf16x2(pw.z) + sum_bf16x2(pw.w));
    l_run = l_run * alpha + psum;
    m_run = m_new;
    const bf16x8 pop = __builtin_bit_cast(bf16x8, pw);
    if (k_begin + kPageTokens * (j + 2) > cd.len) {
      // Last page pair of the conversation: zero V of keys >= len so nothing past the end leaks.
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        va[t].x = mask_bf16x2(va[t].x, key_a + 0 < cd.len, key_a + 1 < cd.len);
        va[t].y = mask_bf16x2(va[t].y, key_a + 2 < cd.len, key_a + 3 < cd.len);
        vb[t].x = mask_bf16x2(vb[t].x, key_a + 16 < cd.len, key_a + 17 < cd.len);
        vb[t].y = mask_bf16x2(vb[t].y, key_a + 18 < cd.len, key_a + 19 < cd.len);
      }
    }
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      o[t] *= alpha;
      o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(va[t], vb[t]), pop, o[t], 0, 0, 0);
    }
  }
  // l_run holds this lane's keys only; sum over the four k-blocks of the column.
  l_run += xor_shfl(l_run, 16);
  l_run += xor_shfl(l_run, 32);
  // A wave past the conversation's end has m = -inf, l = 0, o = 0 and adds nothing below.
  if (wave > 0 && c < a.group) {
    float* x = xch + ((wave - 1) * 8 + c) * (D + 2);
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) x[16 * t + 4 * qd + r] = o[t][r];
    if (qd == 0) {
      x[D] = m_run;
      x[D + 1] = l_run;
    }
  }
  __syncthreads();
  if (wave == 0 && valid && c < a.group) {
    // wave 0 always holds keys, so M is finite; merge in the order w = 0, 1, ...
    float M = m_run;
#pragma unroll
    for (int w = 1; w < kDecodeSubSplits; ++w) M = fmaxf(M, xch[((w - 1) * 8 + c) * (D + 2) + D]);
    const float a0 = fast_exp2(m_run - M);
    float l = l_run * a0;
#pragma unroll
    for (int t = 0; t < DT; ++t) o[t] *= a0;
#pragma unroll
    for (int w = 1; w < kDecodeSubSplits; ++w) {
      const float* x = xch + ((w - 1) * 8 + c) * (D + 2);
      const float aw = fast_exp2(x[D] - M);
      l = __builtin_fmaf(aw, x[D + 1], l);
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) o[t][r] = __builtin_fmaf(aw, x[16 * t + 4 * qd + r], o[t][r]);
    }
    if (a.direct) {  // the item is the whole conversation: out = o / l (as the merge computes it)
      uint16_t* orow = a.out + (static_cast<size_t>(conv_idx) * a.n_kv_heads * a.group + g * a.group + c) * D;
#pragma unroll
      for (int t = 0; t < DT; ++t)
        st8(orow + 16 * t + 4 * qd, make_uint2(pack_bf16x2(o[t][0] / l, o[t][1] / l),
                                               pack_bf16x2(o[t][2] / l, o[t][3] / l)));
      return;
    }
    // non-temporal: the record is read once, by the merge (about 1% faster than plain stores)
    float* pp = a.partials + ((static_cast<size_t>(item) * a.n_kv_heads + g) * a.group + c) * partial_floats(D);
#pragma unroll
    for (int t = 0; t < DT; ++t) __builtin_nontemporal_store(o[t], reinterpret_cast<f32x4*>(pp + 16 * t + 4 * qd));
    if (qd == 0) {
      pp[D] = M;
      pp[D + 1] = l;
    }
  }
}

inline DecodeArgs make_decode_args(const PoolGeom& g, int layer, const DecodeConvDesc* d_convs,
                                   const int32_t* d_order, int n_convs, int n_items, int split_tokens,
                                   const void* q, void* out, const float* partials) {
  DecodeArgs a;
  a.pool = static_cast<const uint16_t*>(g.pool);
  a.n_pages = g.n_pages;
  a.n_kv_heads = g.n_kv_heads;
  a.group = g.n_q_heads / g.n_kv_heads;
  a.layer = layer;
  a.page_table = g.page_table;
  a.max_pages = g.max_pages;
  a.convs = d_convs;
  a.order = d_order;
  a.n_convs = n_convs;
  a.n_items = n_items;
  a.split = split_tokens;
  a.q = static_cast<const uint16_t*>(q);
  a.out = static_cast<uint16_t*>(out);
  a.partials = const_cast<float*>(partials);
  a.direct = 0;
  a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(g.head_dim)));
  return a;
}

}  // namespace cs
