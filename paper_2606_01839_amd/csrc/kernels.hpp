// Host-callable launchers of the gfx950 kernels (defined in the .hip files).
#pragma once

#include <hip/hip_runtime.h>

#include "host/host_state.hpp"

namespace cs {

struct PoolGeom {
  void* pool;          // device base of the KV pool
  int64_t n_pages;
  int n_layers;
  int n_kv_heads;
  int n_q_heads;
  int head_dim;
  int32_t* page_table;  // device mirror [max_convs][max_pages]
  int max_pages;
};

// KV append / unpack: write chunks (see PageChunk) of k,v [n_layers][src_rows][Hkv][D].
hipError_t launch_append(const PoolGeom& g, const PageChunk* d_chunks, int n_chunks, const void* k,
                         const void* v, int64_t src_rows, hipStream_t stream);

// Pack: conversation pages (page-table row `slot`) -> wire [layer][lpage][head] blocks.
hipError_t launch_pack(const PoolGeom& g, int slot, int64_t len, void* wire, hipStream_t stream);

// Unpack: wire logical pages [lp0, lp0 + n_lp) -> physical pages d_pages[0..n_lp) of the
// conversation in page-table row `slot` (length len).
hipError_t launch_unpack(const PoolGeom& g, const void* wire, const int32_t* d_pages, int slot,
                         int64_t len, int lp0, int n_lp, hipStream_t stream);

// Decode partial record of one (work item, query head): o[d], running max m, sum l, two unused
// floats, so records stay 16-byte aligned.
constexpr int partial_floats(int head_dim) { return head_dim + 4; }

// Decode: split kernel over plan items (partials), then the merge kernel (output). d_order: the
// plan's launch order of its n_items items (a permutation).
// direct_out != nullptr (only when every conversation is one item, n_items == n_convs): the split
// writes the final output there and no merge follows.
hipError_t launch_decode_split(const PoolGeom& g, int layer, const DecodeConvDesc* d_convs,
                               const int32_t* d_order, int n_convs, int n_items, int split_tokens, const void* q,
                               float* partials, void* direct_out, hipStream_t stream);
hipError_t launch_decode_merge(const PoolGeom& g, const DecodeConvDesc* d_convs, int n_convs,
                               const float* partials, void* out, hipStream_t stream);
// Merge of layer l (merge_partials -> merge_out) and split of layer split_layer (-> split_partials,
// a different buffer) in one launch; the same conversations and plan for both.
hipError_t launch_decode_merge_split(const PoolGeom& g, int split_layer, const DecodeConvDesc* d_convs,
                                     const int32_t* d_order, int n_convs, int n_items, int split_tokens, const void* q,
                                     float* split_partials, const float* merge_partials,
                                     void* merge_out, hipStream_t stream);

// Streaming-read probe: read `bytes` (a multiple of 16) of device memory once with non-temporal
// 16-byte loads on 8 workgroups per CU; `sink` is 4 bytes of device memory (almost never written).
hipError_t launch_stream_read_probe(const void* src, size_t bytes, uint32_t* sink, int n_cus,
                                    hipStream_t stream);

// Capacity of the static decode scratch (floats): 16 MiB on each GPU.
constexpr size_t kStaticScratchFloats = size_t(4) << 20;
// Device address of the static decode scratch on the current device (looked up once per device
// with hipGetSymbolAddress and cached; allocates nothing).
hipError_t static_decode_scratch(float** out);

// One layer of a mixed step in one launch (head_dim 128 only): the extend tiles of the layer and
// its decode split (partials; the merge follows as launch_decode_merge).
hipError_t launch_mixed_layer(const PoolGeom& g, int layer, const ExtendConvDesc* d_ext_convs,
                              const ExtendTile* d_tiles, int n_tiles, const void* q_ext,
                              void* out_ext, const DecodeConvDesc* d_dec_convs,
                              const int32_t* d_dec_order, int n_dec_convs,
                              int n_items, int split_tokens, const void* q_dec, float* partials,
                              void* direct_out, hipStream_t stream);

// Query tokens per extend/prefill work tile for this head size and GQA group (the host plan must
// match).
int extend_query_tile(int head_dim, int group);

// Extend / prefill: one workgroup per (tile, kv head).
hipError_t launch_extend(const PoolGeom& g, int layer, const ExtendConvDesc* d_convs,
                         const ExtendTile* d_tiles, int n_tiles, const void* q, void* out,
                         hipStream_t stream);

}  // namespace cs
