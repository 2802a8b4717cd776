// Batched single-token decode attention over paged KV (split-K "flash decoding").
//
// Work item = (conversation, logical split of `split` keys, kv head): one wave reads the split's
// pages once and serves all G query heads of the kv head. The two contractions per page pair are
// done on the matrix cores with v_mfma_f32_16x16x32_bf16, the GQA group as the 16-wide N side:
//   S^T[key][head] = K[key][:] . Q[head][:]          (A = K rows straight from the page,
//                                                     B = Q, 8 consecutive dims per lane)
//   O^T[dim][head] += V^T[dim][key] . P^T[key][head]  (A = V^T rows from the page,
//                                                     B = P from the S^T accumulator registers)
// so K and V^T are used in the layout they are stored in (no LDS): each K operand load reads one
// 1 KiB sub-block of a page, each V^T load 512 consecutive bytes.
// The softmax is online in fp32 (exp2 with log2(e)/sqrt(d) folded into the score scale); the
// per-item partial (o, m, l) goes to a workspace and a second kernel merges the splits of each
// (conversation, query head) in a fixed order. No atomics: bitwise deterministic, and split
// boundaries are logical positions, so results do not depend on physical page placement.
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
  int n_items;
  int split;  // keys per split, multiple of 32, <= 1024
  const uint16_t* q;
  uint16_t* out;
  float* partials;  // [n_items * n_kv_heads][group] records of partial_floats(D)
  float scale_log2;
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

template <int D>
__device__ __forceinline__ void split_body(const DecodeArgs& a, const int block) {
  constexpr int KS = D / 32;  // k-steps of the QK^T contraction
  constexpr int DT = D / 16;  // 16-dim tiles of the output
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int work = block * 4 + wave;  // = item * n_kv_heads + kv head
  if (work >= a.n_items * a.n_kv_heads) return;
  const int item = work / a.n_kv_heads, g = work % a.n_kv_heads;
  const auto* convs = as_const(a.convs);
  const int conv_idx = find_conv(convs, a.n_convs, item);
  const DecodeConvDesc cd = load_desc(convs + conv_idx);
  const int k_begin = (item - cd.item_start) * a.split;
  const int k_end = min(cd.len, k_begin + a.split);
  const int n_pg = (k_end - k_begin + kPageTokens - 1) / kPageTokens;
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
  if (c < a.group) {
    float* pp = a.partials + (static_cast<size_t>(work) * a.group + c) * partial_floats(D);
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) pp[16 * t + 4 * qd + r] = o[t][r];
    if (qd == 0) {
      pp[D] = m_run;
      pp[D + 1] = l_run;
    }
  }
}

// One workgroup per (conversation, query head): log-sum-exp merge of its splits, in three steps
// whose order depends only on the split count (bitwise deterministic): the maximum M of the split
// maxima; per thread, the weighted sum over a fixed subset of the splits (split group sg = thread /
// (D/4) takes splits sg, sg + SG, ...; dim group = 4 consecutive dims, one 16-byte load); then the
// split groups added in order 0 .. SG-1.
template <int D>
__device__ __forceinline__ void merge_body(const DecodeArgs& a, const int b, const int h) {
  constexpr int DV = D / 4;          // dim groups (4 dims each)
  constexpr int SG = 256 / DV;       // split groups
  constexpr int R = partial_floats(D);
  __shared__ float red_o[SG][D];
  __shared__ float red_l[SG];
  __shared__ float wave_max[4];
  const int g = h / a.group, c = h % a.group;
  const DecodeConvDesc cd = load_desc(as_const(a.convs) + b);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t split_stride = static_cast<size_t>(a.n_kv_heads) * a.group * R;
  const float* base =
      a.partials + ((static_cast<size_t>(cd.item_start) * a.n_kv_heads + g) * a.group + c) * R;
  const int n = cd.n_splits;

  float M = -INFINITY;
  for (int s = tid; s < n; s += 256) M = fmaxf(M, base[s * split_stride + D]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, xor_shfl(M, off));
  if (lane == 0) wave_max[wave] = M;
  __syncthreads();
  M = fmaxf(fmaxf(wave_max[0], wave_max[1]), fmaxf(wave_max[2], wave_max[3]));

  const int dg = tid % DV, sg = tid / DV;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
#pragma unroll 4
  for (int s = sg; s < n; s += SG) {
    const float* p = base + s * split_stride;
    const f32x2 ml = *reinterpret_cast<const f32x2*>(p + D);
    const f32x4 v = *reinterpret_cast<const f32x4*>(p + 4 * dg);
    const float w = fast_exp2(ml.x - M);
    acc += w * v;
    den += w * ml.y;
  }
  *reinterpret_cast<f32x4*>(&red_o[sg][4 * dg]) = acc;
  if (dg == 0) red_l[sg] = den;
  __syncthreads();
  if (tid < D) {
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int k = 0; k < SG; ++k) {
      o += red_o[k][tid];
      l += red_l[k];
    }
    uint16_t* orow = a.out + (static_cast<size_t>(b) * a.n_kv_heads * a.group + h) * D;
    orow[tid] = static_cast<uint16_t>(pack_bf16x2(o / l, 0.f) & 0xFFFFu);
  }
}

template <int D>
__global__ __launch_bounds__(256) void decode_split_kernel(DecodeArgs a) { split_body<D>(a, blockIdx.x); }

template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeArgs a) {
  merge_body<D>(a, blockIdx.x, blockIdx.y);
}

// The merge of one layer and the split of the next in one launch (a multi-layer step): the first
// n_conv * n_q_heads workgroups merge layer l's partials (buffer am.partials), the others run layer
// l+1's split into the other partial buffer. Saves one launch and its gap per layer.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_split_kernel(DecodeArgs am, DecodeArgs as) {
  const int n_merge = am.n_convs * am.n_kv_heads * am.group;
  const int blk = blockIdx.x;
  if (blk < n_merge) {
    const int nqh = am.n_kv_heads * am.group;
    merge_body<D>(am, blk / nqh, blk % nqh);
  } else {
    split_body<D>(as, blk - n_merge);
  }
}

static DecodeArgs make_args(const PoolGeom& g, int layer, const DecodeConvDesc* d_convs, int n_convs,
                            int n_items, int split_tokens, const void* q, void* out,
                            const float* partials) {
  DecodeArgs a;
  a.pool = static_cast<const uint16_t*>(g.pool);
  a.n_pages = g.n_pages;
  a.n_kv_heads = g.n_kv_heads;
  a.group = g.n_q_heads / g.n_kv_heads;
  a.layer = layer;
  a.page_table = g.page_table;
  a.max_pages = g.max_pages;
  a.convs = d_convs;
  a.n_convs = n_convs;
  a.n_items = n_items;
  a.split = split_tokens;
  a.q = static_cast<const uint16_t*>(q);
  a.out = static_cast<uint16_t*>(out);
  a.partials = const_cast<float*>(partials);
  a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(g.head_dim)));
  return a;
}

hipError_t launch_decode_split(const PoolGeom& g, int layer, const DecodeConvDesc* d_convs,
                               int n_convs, int n_items, int split_tokens, const void* q,
                               float* partials, hipStream_t stream) {
  if (n_convs == 0) return hipSuccess;
  const DecodeArgs a = make_args(g, layer, d_convs, n_convs, n_items, split_tokens, q, nullptr, partials);
  const int blocks = (n_items * g.n_kv_heads + 3) / 4;
  if (g.head_dim == 128) decode_split_kernel<128><<<blocks, 256, 0, stream>>>(a);
  else if (g.head_dim == 64) decode_split_kernel<64><<<blocks, 256, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_decode_merge_split(const PoolGeom& g, int split_layer, const DecodeConvDesc* d_convs,
                                     int n_convs, int n_items, int split_tokens, const void* q,
                                     float* split_partials, const float* merge_partials,
                                     void* merge_out, hipStream_t stream) {
  if (n_convs == 0) return hipSuccess;
  const DecodeArgs as = make_args(g, split_layer, d_convs, n_convs, n_items, split_tokens, q, nullptr,
                                  split_partials);
  const DecodeArgs am = make_args(g, 0, d_convs, n_convs, 0, 0, nullptr, merge_out, merge_partials);
  const int blocks = n_convs * g.n_q_heads + (n_items * g.n_kv_heads + 3) / 4;
  if (g.head_dim == 128) decode_merge_split_kernel<128><<<blocks, 256, 0, stream>>>(am, as);
  else if (g.head_dim == 64) decode_merge_split_kernel<64><<<blocks, 256, 0, stream>>>(am, as);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_decode_merge(const PoolGeom& g, const DecodeConvDesc* d_convs, int n_convs,
                               const float* partials, void* out, hipStream_t stream) {
  if (n_convs == 0) return hipSuccess;
  const DecodeArgs a = make_args(g, 0, d_convs, n_convs, 0, 0, nullptr, out, partials);
  const dim3 grid(n_convs, g.n_q_heads);
  if (g.head_dim == 128) decode_merge_kernel<128><<<grid, 256, 0, stream>>>(a);
  else if (g.head_dim == 64) decode_merge_kernel<64><<<grid, 256, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace cs
