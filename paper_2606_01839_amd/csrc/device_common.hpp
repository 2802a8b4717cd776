// Device-side helpers shared by the gfx950 kernels: vector types, the pool block layout, bf16
// conversions, cross-lane reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cs {

constexpr int kPageTokens = 16;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Pool block of (layer, page, kv head), bf16: the K part, then V^T[D][16] (dimension-major). The
// K part is D/32 sub-blocks of 32 dims, each K[16 tokens][32 dims] token-major: the 64-byte pieces
// of one 32-dim range of all 16 keys are 1 KiB of consecutive bytes, which is what one 16-byte-
// per-lane load of the matrix-core K operand (16 keys x 4 lanes) reads. Offsets in elements.
template <int D>
__device__ __forceinline__ size_t block_elem(int layer, int page, int head, int64_t n_pages,
                                             int n_kv_heads) {
  return ((static_cast<size_t>(layer) * static_cast<size_t>(n_pages) + static_cast<size_t>(page)) *
              static_cast<size_t>(n_kv_heads) +
          static_cast<size_t>(head)) *
         static_cast<size_t>(2 * kPageTokens * D);
}

// Element offset inside a block of dims 8 chunk .. 8 chunk + 7 of token t (K part).
__device__ __forceinline__ int k_elem(int t, int chunk) {
  return ((chunk >> 2) * kPageTokens + t) * 32 + (chunk & 3) * 8;
}

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ uint2 ld8(const void* p) { return *reinterpret_cast<const uint2*>(p); }
__device__ __forceinline__ void st16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }
// Streaming loads of data read exactly once (K/V in decode, pool blocks in pack/unpack): the
// non-temporal hint (global_load ... nt) keeps them from displacing reused lines in the caches;
// on MI355X a stream of such 16-byte loads reads HBM about 10% faster than plain loads.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 ld16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 ld8_nt(const void* p) {
  const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
  return make_uint2(v.x, v.y);
}
// Streaming store of data no kernel of the same pass reads back (wire buffer, freshly placed pages).
__device__ __forceinline__ void st16_nt(void* p, uint4 v) {
  const u32x4_t x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t*>(p));
}
__device__ __forceinline__ void st8(void* p, uint2 v) { *reinterpret_cast<uint2*>(p) = v; }

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ bf16x8 as_bf16x8(uint2 a, uint2 b) {
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// fp32 pair -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// Sum of the two bf16 values packed in w, in fp32 (exact upcasts).
__device__ __forceinline__ float sum_bf16x2(uint32_t w) {
  return __uint_as_float(w << 16) + __uint_as_float(w & 0xFFFF0000u);
}

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Keep the bf16 halves of a 32-bit word selected by keep_lo / keep_hi, zero the others.
__device__ __forceinline__ uint32_t mask_bf16x2(uint32_t w, bool keep_lo, bool keep_hi) {
  return w & ((keep_lo ? 0x0000FFFFu : 0u) | (keep_hi ? 0xFFFF0000u : 0u));
}

// Cross-lane exchange within a wave64 (ds_bpermute); lane ^ mask.
__device__ __forceinline__ float xor_shfl(float v, int mask) {
  int lane = __lane_id();
  return __int_as_float(__builtin_amdgcn_ds_bpermute((lane ^ mask) << 2, __float_as_int(v)));
}

// max / sum of v over lanes l and l ^ 32, returned to both (v_permlane32_swap on gfx950 exchanges
// the two 32-lane halves; each lane sees {v[l], v[l ^ 32]} in its two results, whatever their order).
__device__ __forceinline__ float halves_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace cs
