// Batched single-token decode attention over paged KV (split-K "flash decoding").
//
// A work item is up to kDecodeSubSplits splits (`split` keys each) of consecutive keys of one
// (conversation, kv head), taken by one workgroup; its waves share its keys evenly, each reading
// its range once and serving all G query heads of the kv head. Workgroups take the items in the
// plan's launch order (full items first, then shorter ones). The two contractions per page pair are done on the matrix cores with
// v_mfma_f32_16x16x32_bf16, the GQA group as the 16-wide N side:
//   S^T[key][head] = K[key][:] . Q[head][:]          (A = K rows straight from the page,
//                                                     B = Q, 8 consecutive dims per lane)
//   O^T[dim][head] += V^T[dim][key] . P^T[key][head]  (A = V^T rows from the page,
//                                                     B = P from the S^T accumulator registers)
// so K and V^T are used in the layout they are stored in: each K operand load reads one 1 KiB
// sub-block of a page, each V^T load 512 consecutive bytes. The softmax is online in fp32 (exp2
// with log2(e)/sqrt(d) folded into the score scale). The waves of an item merge their (o, m, l) in
// LDS and write one partial record per (item, query head) to a workspace (decode_split.hpp); a
// second kernel merges the items of each (conversation, query head). Both merges run in a fixed
// order and there are no atomics: bitwise deterministic, and split boundaries are logical
// positions, so results do not depend on physical page placement.
#include <cmath>
#include <mutex>

#include "decode_split.hpp"

namespace cs {

namespace {
// Static decode scratch of the allocation-free decode entry point: the split partial records live
// here instead of in the pool's workspace. Each GPU the library runs on holds its own copy until
// the process ends. Host code never passes `scratch` itself to a kernel (on the host it is only a
// stand-in symbol): its device address, per device, comes from hipGetSymbolAddress below.
__device__ __align__(256) float scratch[kStaticScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_dev[kMaxDevices] = {};
}  // namespace

hipError_t static_decode_scratch(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // with `dev` current: this device's copy
    if (e != hipSuccess) return e;
    g_scratch_dev[dev] = static_cast<float*>(p);
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

// Log-sum-exp merge of the item records of one (conversation b, query head h) by 256 threads (`tid`
// in 0 .. 255, LDS `lds`), in three steps whose order depends only on the record count (bitwise
// deterministic): the maximum M of the record maxima; per thread, the weighted sum over a fixed
// subset of the records (group sg = tid / (D/4) takes records sg, sg + SG, ...; dim group = 4
// consecutive dims, one 16-byte load); then the groups added in order 0 .. SG-1. With valid =
// false the threads only pass the two barriers.
template <int D>
struct MergeLds {
  float red_o[256 / (D / 4)][D];
  float red_l[256 / (D / 4)];
  float wave_max[4];
};

template <int D>
__device__ __forceinline__ void merge_body(const DecodeArgs& a, const int b, const int h, const int tid,
                                           MergeLds<D>& lds, const bool valid) {
  constexpr int DV = D / 4;          // dim groups (4 dims each)
  constexpr int SG = 256 / DV;       // record groups
  constexpr int R = partial_floats(D);
  const int g = h / a.group, c = h % a.group;
  const DecodeConvDesc cd = load_desc(as_const(a.convs) + (valid ? b : 0));
  const int lane = tid & 63, wave = tid >> 6;
  const size_t split_stride = static_cast<size_t>(a.n_kv_heads) * a.group * R;
  const float* base =
      a.partials + ((static_cast<size_t>(cd.item_start) * a.n_kv_heads + g) * a.group + c) * R;
  const int n = valid ? cd.n_splits : 0;

  float M = -INFINITY;
  for (int s = tid; s < n; s += 256) M = fmaxf(M, base[s * split_stride + D]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, xor_shfl(M, off));
  if (lane == 0) lds.wave_max[wave] = M;
  __syncthreads();
  M = fmaxf(fmaxf(lds.wave_max[0], lds.wave_max[1]), fmaxf(lds.wave_max[2], lds.wave_max[3]));

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
  *reinterpret_cast<f32x4*>(&lds.red_o[sg][4 * dg]) = acc;
  if (dg == 0) lds.red_l[sg] = den;
  __syncthreads();
  if (valid && tid < D) {
    float o = 0.f, l = 0.f;
#pragma unroll
    for (int k = 0; k < SG; ++k) {
      o += lds.red_o[k][tid];
      l += lds.red_l[k];
    }
    uint16_t* orow = a.out + (static_cast<size_t>(b) * a.n_kv_heads * a.group + h) * D;
    orow[tid] = static_cast<uint16_t>(pack_bf16x2(o / l, 0.f) & 0xFFFFu);
  }
}

template <int D>
__global__ __launch_bounds__(kDecodeItemThreads) void decode_split_kernel(DecodeArgs a) {
  __shared__ float xch[split_exchange_floats<D>()];
  split_body<D>(a, blockIdx.x, __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), xch);
}

template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(DecodeArgs a) {
  __shared__ MergeLds<D> lds;
  merge_body<D>(a, blockIdx.x, blockIdx.y, threadIdx.x, lds, true);
}

// The merge of one layer and the split of the next in one launch (a multi-layer step): the first
// workgroups merge layer l's partials (buffer am.partials), kDecodeItemThreads / 256 (conversation,
// query head) pairs each, the others run layer l+1's split into the other partial buffer. Saves
// one launch and its gap per layer.
template <int D>
__global__ __launch_bounds__(kDecodeItemThreads) void decode_merge_split_kernel(DecodeArgs am, DecodeArgs as,
                                                                                int merge_blocks) {
  constexpr int kPerBlock = kDecodeItemThreads / 256;
  __shared__ float xch[split_exchange_floats<D>()];
  __shared__ MergeLds<D> lds[kPerBlock];
  const int blk = blockIdx.x;
  if (blk < merge_blocks) {
    const int nqh = am.n_kv_heads * am.group;
    const int part = threadIdx.x >> 8, pair = blk * kPerBlock + part;
    const bool valid = pair < am.n_convs * nqh;
    merge_body<D>(am, valid ? pair / nqh : 0, valid ? pair % nqh : 0, threadIdx.x & 255, lds[part], valid);
  } else {
    split_body<D>(as, blk - merge_blocks, __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), xch);
  }
}

hipError_t launch_decode_split(const PoolGeom& g, int layer, const DecodeConvDesc* d_convs,
                               const int32_t* d_order, int n_convs, int n_items, int split_tokens,
                               const void* q, float* partials, void* direct_out, hipStream_t stream) {
  if (n_convs == 0) return hipSuccess;
  if (d_order == nullptr || n_items < n_convs) return hipErrorInvalidValue;
  DecodeArgs a = make_decode_args(g, layer, d_convs, d_order, n_convs, n_items, split_tokens, q, direct_out,
                                  partials);
  a.direct = direct_out != nullptr && n_items == n_convs;
  if (direct_out != nullptr && !a.direct) return hipErrorInvalidValue;
  const int blocks = n_items * g.n_kv_heads;
  if (g.head_dim == 128) decode_split_kernel<128><<<blocks, kDecodeItemThreads, 0, stream>>>(a);
  else if (g.head_dim == 64) decode_split_kernel<64><<<blocks, kDecodeItemThreads, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_decode_merge_split(const PoolGeom& g, int split_layer, const DecodeConvDesc* d_convs,
                                     const int32_t* d_order, int n_convs, int n_items, int split_tokens,
                                     const void* q, float* split_partials, const float* merge_partials,
                                     void* merge_out, hipStream_t stream) {
  if (n_convs == 0) return hipSuccess;
  if (d_order == nullptr || n_items < n_convs) return hipErrorInvalidValue;
  const DecodeArgs as = make_decode_args(g, split_layer, d_convs, d_order, n_convs, n_items, split_tokens, q,
                                         nullptr, split_partials);
  const DecodeArgs am = make_decode_args(g, 0, d_convs, nullptr, n_convs, 0, 0, nullptr, merge_out,
                                         merge_partials);
  constexpr int kPerBlock = kDecodeItemThreads / 256;
  const int merge_blocks = (n_convs * g.n_q_heads + kPerBlock - 1) / kPerBlock;
  const int blocks = merge_blocks + n_items * g.n_kv_heads;
  if (g.head_dim == 128)
    decode_merge_split_kernel<128><<<blocks, kDecodeItemThreads, 0, stream>>>(am, as, merge_blocks);
  else if (g.head_dim == 64)
    decode_merge_split_kernel<64><<<blocks, kDecodeItemThreads, 0, stream>>>(am, as, merge_blocks);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_decode_merge(const PoolGeom& g, const DecodeConvDesc* d_convs, int n_convs,
                               const float* partials, void* out, hipStream_t stream) {
  if (n_convs == 0) return hipSuccess;
  const DecodeArgs a = make_decode_args(g, 0, d_convs, nullptr, n_convs, 0, 0, nullptr, out, partials);
  const dim3 grid(n_convs, g.n_q_heads);
  if (g.head_dim == 128) decode_merge_kernel<128><<<grid, 256, 0, stream>>>(a);
  else if (g.head_dim == 64) decode_merge_kernel<64><<<grid, 256, 0, stream>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace cs
