// KV movement kernels: append new tokens into pages, pack a conversation into the transfer wire
// format, unpack a wire buffer into freshly placed pages. Pure byte movement (bit-exact); every
// one is HBM-bound. A pool block (layer, page, kv head) is its K part (D/32 token-major sub-blocks
// of 32 dims, see k_elem) followed by V^T[D][16] dimension-major; token slots past a
// conversation's end are kept zero. The wire format of the transfer is the same block format.
#include "device_common.hpp"
#include "kernels.hpp"

namespace cs {

// ---------------------------------------------------------------------------------------------
// Append: one wave per (layer, kv head) and kAppendChunks page chunks, up to 4 kv heads per
// workgroup. A wave issues the loads of all its chunks before any store (more bytes in flight per
// wave, half as many waves), copies K pieces with 16-byte accesses, and stages V rows in LDS to
// write them transposed. A chunk that starts a page (t0 = 0) writes the whole page, zeros in slots
// [t1, 16); a chunk that continues a page writes only its slots [t0, t1): the rest of the page is
// already zero, since a page's first chunk always starts at slot 0 (pages are taken as a
// conversation crosses a 16-token boundary) and unpack writes whole pages.
// ---------------------------------------------------------------------------------------------
constexpr int kAppendChunks = 2;

template <int D>
__global__ __launch_bounds__(256) void kv_append_kernel(const PageChunk* __restrict__ chunks,
                                                       int n_chunks,
                                                       const uint16_t* __restrict__ k_src,
                                                       const uint16_t* __restrict__ v_src,
                                                       int64_t src_rows, uint16_t* __restrict__ pool,
                                                       int64_t n_pages, int n_kv_heads,
                                                       int32_t* __restrict__ page_table,
                                                       int max_pages) {
  constexpr int kChunksPerRow = D / 8;            // 16-byte chunks per token row
  constexpr int kRowsPerPass = 64 / kChunksPerRow;
  constexpr int kPasses = kPageTokens / kRowsPerPass;
  constexpr int CH = kAppendChunks;
  __shared__ uint16_t vts[4][CH][kPageTokens][D + 8];

  const int waves = blockDim.x >> 6, wave = threadIdx.x >> 6;
  const int groups = n_kv_heads / waves;  // workgroups per (chunk group, layer)
  const int layer = blockIdx.y / groups;
  const int head = (blockIdx.y % groups) * waves + wave;
  const int lane = threadIdx.x & 63;
  const int ch = lane % kChunksPerRow;

  PageChunk c[CH];
  bool have[CH];
  uint4 kv[CH][kPasses], vv[CH][kPasses];
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int idx = blockIdx.x * CH + i;
    have[i] = idx < n_chunks;
    c[i] = chunks[have[i] ? idx : 0];
#pragma unroll
    for (int ps = 0; ps < kPasses; ++ps) {
      const int t = lane / kChunksPerRow + ps * kRowsPerPass;
      kv[i][ps] = make_uint4(0, 0, 0, 0);
      vv[i][ps] = make_uint4(0, 0, 0, 0);
      if (have[i] && t >= c[i].t0 && t < c[i].t1) {
        const size_t row = static_cast<size_t>(c[i].src_row) + static_cast<size_t>(t - c[i].t0);
        const size_t src =
            ((static_cast<size_t>(layer) * static_cast<size_t>(src_rows) + row) * n_kv_heads + head) *
                D + ch * 8;
        kv[i][ps] = ld16(k_src + src);
        vv[i][ps] = ld16(v_src + src);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    if (!have[i]) continue;
    uint16_t* blk = pool + block_elem<D>(layer, c[i].page, head, n_pages, n_kv_heads);
#pragma unroll
    for (int ps = 0; ps < kPasses; ++ps) {
      const int t = lane / kChunksPerRow + ps * kRowsPerPass;
      if (t >= c[i].t0 && (t < c[i].t1 || c[i].t0 == 0)) st16(blk + k_elem(t, ch), kv[i][ps]);
      *reinterpret_cast<uint4*>(&vts[wave][i][t][ch * 8]) = vv[i][ps];
    }
  }
  __syncthreads();

#pragma unroll
  for (int i = 0; i < CH; ++i) {
    if (!have[i]) continue;
    const auto& vt = vts[wave][i];
    uint16_t* vdst = pool + block_elem<D>(layer, c[i].page, head, n_pages, n_kv_heads) + kPageTokens * D;
#pragma unroll
    for (int e = lane; e < D; e += 64) {
      uint16_t* row = vdst + e * kPageTokens;
      if (c[i].t0 == 0) {
        uint32_t w[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          w[j] = static_cast<uint32_t>(vt[2 * j][e]) | (static_cast<uint32_t>(vt[2 * j + 1][e]) << 16);
        st16(row, make_uint4(w[0], w[1], w[2], w[3]));
        st16(row + 8, make_uint4(w[4], w[5], w[6], w[7]));
      } else {
        for (int t = c[i].t0; t < c[i].t1; ++t) row[t] = vt[t][e];
      }
    }
    if (c[i].new_page && blockIdx.y == 0 && threadIdx.x == 0)
      page_table[static_cast<size_t>(c[i].slot) * max_pages + c[i].lpage] = c[i].page;
  }
}

// Zero the token slots >= valid inside 16-byte chunk i (8 elements) of a block.
template <int D>
__device__ __forceinline__ uint4 mask_tail(uint4 x, int i, int valid) {
  const int e0 = 8 * i;
  if (e0 < kPageTokens * D) {           // K part: chunk i holds dims of token (i % 64) / 4
    return ((i & 63) >> 2) < valid ? x : make_uint4(0, 0, 0, 0);
  }
  const int t0 = (e0 - kPageTokens * D) % kPageTokens;  // V^T part: tokens t0 .. t0+7 of one dim
  x.x = mask_bf16x2(x.x, t0 + 0 < valid, t0 + 1 < valid);
  x.y = mask_bf16x2(x.y, t0 + 2 < valid, t0 + 3 < valid);
  x.z = mask_bf16x2(x.z, t0 + 4 < valid, t0 + 5 < valid);
  x.w = mask_bf16x2(x.w, t0 + 6 < valid, t0 + 7 < valid);
  return x;
}

// ---------------------------------------------------------------------------------------------
// Pack: one wave per (logical page, layer, kv head) block; all of a lane's loads are issued
// before its stores. Tail slots of the last page are written as zeros.
// ---------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void kv_pack_kernel(const uint16_t* __restrict__ pool,
                                                     int64_t n_pages, int n_kv_heads,
                                                     const int32_t* __restrict__ pt_row, int64_t len,
                                                     uint16_t* __restrict__ wire, int n_lpages) {
  constexpr int kChunks = 2 * kPageTokens * D / 8;  // 16-byte chunks per block
  constexpr int kPerLane = kChunks / 64;
  const int lp = blockIdx.x;
  const int layer = blockIdx.y / n_kv_heads, head = blockIdx.y % n_kv_heads;
  const int page = pt_row[lp];
  const uint16_t* src = pool + block_elem<D>(layer, page, head, n_pages, n_kv_heads);
  uint16_t* dst = wire + ((static_cast<size_t>(layer) * n_lpages + lp) * n_kv_heads + head) *
                             static_cast<size_t>(2 * kPageTokens * D);
  const int64_t rem = len - static_cast<int64_t>(lp) * kPageTokens;
  const int valid = rem < kPageTokens ? static_cast<int>(rem) : kPageTokens;
  uint4 x[kPerLane];
#pragma unroll
  for (int j = 0; j < kPerLane; ++j) x[j] = ld16_nt(src + 8 * (threadIdx.x + 64 * j));
#pragma unroll
  for (int j = 0; j < kPerLane; ++j) {
    const int i = threadIdx.x + 64 * j;
    st16_nt(dst + 8 * i, valid < kPageTokens ? mask_tail<D>(x[j], i, valid) : x[j]);
  }
}

// ---------------------------------------------------------------------------------------------
// Unpack: inverse of pack into pages d_pages[lp]; also fills the page-table mirror row.
// ---------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void kv_unpack_kernel(const uint16_t* __restrict__ wire,
                                                       const int32_t* __restrict__ d_pages,
                                                       int64_t len, uint16_t* __restrict__ pool,
                                                       int64_t n_pages, int n_kv_heads,
                                                       int32_t* __restrict__ pt_row, int n_lpages,
                                                       int lp0) {
  constexpr int kChunks = 2 * kPageTokens * D / 8;
  constexpr int kPerLane = kChunks / 64;
  const int lp = lp0 + blockIdx.x;
  const int layer = blockIdx.y / n_kv_heads, head = blockIdx.y % n_kv_heads;
  const int page = d_pages[blockIdx.x];
  const uint16_t* src = wire + ((static_cast<size_t>(layer) * n_lpages + lp) * n_kv_heads + head) *
                                   static_cast<size_t>(2 * kPageTokens * D);
  uint16_t* dst = pool + block_elem<D>(layer, page, head, n_pages, n_kv_heads);
  const int64_t rem = len - static_cast<int64_t>(lp) * kPageTokens;
  const int valid = rem < kPageTokens ? static_cast<int>(rem) : kPageTokens;
  uint4 x[kPerLane];
#pragma unroll
  for (int j = 0; j < kPerLane; ++j) x[j] = ld16_nt(src + 8 * (threadIdx.x + 64 * j));
#pragma unroll
  for (int j = 0; j < kPerLane; ++j) {
    const int i = threadIdx.x + 64 * j;
    st16_nt(dst + 8 * i, valid < kPageTokens ? mask_tail<D>(x[j], i, valid) : x[j]);
  }
  if (blockIdx.y == 0 && threadIdx.x == 0) pt_row[lp] = page;
}

// ---------------------------------------------------------------------------------------------
template <typename F>
static hipError_t by_dim(int D, F&& f) {
  if (D == 64) return f(std::integral_constant<int, 64>{});
  if (D == 128) return f(std::integral_constant<int, 128>{});
  return hipErrorInvalidValue;
}

hipError_t launch_append(const PoolGeom& g, const PageChunk* d_chunks, int n_chunks, const void* k,
                         const void* v, int64_t src_rows, hipStream_t stream) {
  if (n_chunks == 0) return hipSuccess;
  return by_dim(g.head_dim, [&](auto dc) {
    constexpr int D = decltype(dc)::value;
    // kv heads per workgroup: 4, 2 or 1, whichever is the largest that divides n_kv_heads
    const int waves = g.n_kv_heads % 4 == 0 ? 4 : (g.n_kv_heads % 2 == 0 ? 2 : 1);
    dim3 grid((n_chunks + kAppendChunks - 1) / kAppendChunks, g.n_layers * (g.n_kv_heads / waves));
    kv_append_kernel<D><<<grid, 64 * waves, 0, stream>>>(
        d_chunks, n_chunks, static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), src_rows,
        static_cast<uint16_t*>(g.pool), g.n_pages, g.n_kv_heads, g.page_table, g.max_pages);
    return hipGetLastError();
  });
}

hipError_t launch_pack(const PoolGeom& g, int slot, int64_t len, void* wire, hipStream_t stream) {
  const int n_lpages = static_cast<int>(pages_for(len));
  if (n_lpages == 0) return hipSuccess;
  return by_dim(g.head_dim, [&](auto dc) {
    constexpr int D = decltype(dc)::value;
    dim3 grid(n_lpages, g.n_layers * g.n_kv_heads);
    kv_pack_kernel<D><<<grid, 64, 0, stream>>>(
        static_cast<const uint16_t*>(g.pool), g.n_pages, g.n_kv_heads,
        g.page_table + static_cast<size_t>(slot) * g.max_pages, len, static_cast<uint16_t*>(wire),
        n_lpages);
    return hipGetLastError();
  });
}

hipError_t launch_unpack(const PoolGeom& g, const void* wire, const int32_t* d_pages, int slot,
                         int64_t len, int lp0, int n_lp, hipStream_t stream) {
  const int n_lpages = static_cast<int>(pages_for(len));
  if (n_lp == 0) return hipSuccess;
  return by_dim(g.head_dim, [&](auto dc) {
    constexpr int D = decltype(dc)::value;
    dim3 grid(n_lp, g.n_layers * g.n_kv_heads);
    kv_unpack_kernel<D><<<grid, 64, 0, stream>>>(
        static_cast<const uint16_t*>(wire), d_pages, len, static_cast<uint16_t*>(g.pool),
        g.n_pages, g.n_kv_heads, g.page_table + static_cast<size_t>(slot) * g.max_pages, n_lpages,
        lp0);
    return hipGetLastError();
  });
}

}  // namespace cs
