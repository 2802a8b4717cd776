// Turn-1 prefill and turn-N extend-prefill attention over paged KV (flash-attention forward).
//
// A workgroup owns one (conversation, query block, kv head) tile; its waves cover the G query
// heads of that kv head (the GQA group), so every K/V tile in LDS serves all the query rows of
// the group (256 rows at head_dim 128).
// Each wave computes the transposed score tile on the matrix cores (v_mfma_f32_32x32x16_bf16):
//   S^T[key][query] = K[key][:] . Q[query][:]       A = K rows from LDS, B = Q kept in registers
//   O^T[dim][query] += V^T[dim][key] . P^T[key][query]   A = V^T rows from LDS, B = P registers
// With the transposed formulation every lane owns one query row (32 rows of a 32x32 tile, the two
// 32-lane halves holding different keys), so the online-softmax max/sum are in-lane except for
// one exchange between the halves, and the P accumulator registers are directly the B operand of
// the PV product: the key order of K or V^T in LDS is arranged so the two contractions agree.
//
// head_dim 128 (attn_fwd_kernel): eight waves, G query heads x 8/G blocks of 32 queries (a 64-query
// tile at G = 4, 128 queries at G = 2), two waves per SIMD.
// K/V tiles of 64 keys (4 pages) are copied from HBM straight into a four-deep LDS ring with
// global_load_lds_dwordx4 (no staging registers, no LDS store instructions), three tiles ahead;
// the K operands of tile j+1 are read into registers while the PV product of tile j runs.
// head_dim 64 (attn_fwd_staged_kernel): one wave per query head (64 queries in two 32-row tiles),
// one wave per SIMD; K/V tiles staged through registers into a double-buffered LDS tile two tiles
// ahead. In both, diagonal tiles apply the causal mask and fully visible tiles skip it.
#include <cmath>

#include "decode_split.hpp"
#include "device_common.hpp"
#include "kernels.hpp"

namespace cs {

struct ExtendArgs {
  const uint16_t* pool;
  int64_t n_pages;
  int n_kv_heads;
  int layer;
  const int32_t* page_table;
  int max_pages;
  const ExtendConvDesc* convs;
  const ExtendTile* tiles;
  const uint16_t* q;
  uint16_t* out;
  float scale_log2;
};

constexpr int kBN = 64;  // keys per tile
constexpr int kBM = 64;  // query tokens per workgroup of the head_dim 64 kernel

// LDS tile of the staged kernel (padded rows: bank-conflict-free MFMA operand reads).
template <int D>
struct FwdSmem {
  static constexpr int kRowK = D + 8;    // K tile row stride (elements), padded
  static constexpr int kRowV = kBN + 8;  // V^T tile row stride (elements), padded
  uint16_t k[2][kBN][kRowK];
  uint16_t v[2][D][kRowV];
};

// Position of key group c (4 keys) of a 16-key group inside the permuted V^T row:
// groups hold keys {0-3, 8-11, 4-7, 12-15} so that 32-lane half h reads keys {4h..4h+3, 8+4h..}
// as one 16-byte run.
__device__ __forceinline__ int vt_group_pos(int c) { return ((c & 1) << 1) | (c >> 1); }

// Lazy rescaling threshold (log2 units): the running max used in the exponent is only raised when
// a new score exceeds it by more than this, so P <= 2^8 and the O/l rescale is rare.
constexpr float kRescaleLog2 = 8.f;
// Per-lane bound on the sum of a tile's weights (32 keys per lane) before the max is refreshed.
constexpr float kSumLimit = 256.f;

// ------------------------------------------------------------------------------------------------
// head_dim 128: K/V copied from HBM straight into LDS.
// LDS ring of four tiles: the K parts of the four buffers in the low 64 KiB (16 KiB each), their
// V^T parts in the high 64 KiB, so every operand read reaches its buffer through the instruction's
// 16-bit offset field (no address arithmetic per read). K as 64 rows x 256 B, the 16-byte chunk
// index XOR-swizzled by the row (chunk ^ (row & 15)); V^T page by page, 128 dims x 32 B (16 keys)
// per page, the two
// 16-byte halves of a dim swapped when bit 2 xor bit 3 of the dim is set. A 16-byte operand read
// is served 16 lanes at a time over 256 bytes of banks: the 16 rows (K) or dims (V^T) such a group
// reads then fall in 16 distinct 16-byte bank groups (rocprofv3 SQ_LDS_BANK_CONFLICT = 0), while
// every copy instruction still writes 1 KiB of consecutive LDS bytes.
// ------------------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p));
}
// Copy 16 bytes per lane from global memory (wave-uniform base + per-lane byte offset) straight
// into LDS: lane l writes LDS bytes lds + 16 l .. +15 (global_load_lds_dwordx4, destination base in
// M0). The copy is tracked by the vector-memory counter only; M0 is saved and restored around it.
__device__ __forceinline__ void dma16(uint32_t lds, const void* gbase, uint32_t voff) {
  uint32_t saved;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %2, %3\n\ts_mov_b32 m0, %0"
               : "=&s"(saved) : "s"(lds), "v"(voff), "s"(gbase) : "memory");
}
// Wait until at most N of this wave's vector-memory operations (its copies) are in flight, then a
// workgroup barrier: afterwards every wave's copies issued before its own last N have landed.
template <int N>
__device__ __forceinline__ void dma_wait_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" :: "n"(N) : "memory");
}

// One (tile, kv head) workgroup of the head_dim 128 kernel (`block` = its index in the grid).
template <int G>
__device__ __forceinline__ void attn_fwd_block(const ExtendArgs& a, const int block) {
  constexpr int D = 128;
  constexpr int NW = 8;                   // waves: G query heads x (8 / G) blocks of 32 queries
  constexpr int BM = 32 * (NW / G);       // queries per workgroup
  static_assert(NW % G == 0, "the group must divide the eight waves");
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  constexpr int NB = 16;                  // 1 KiB blocks per K (and per V^T) tile
  constexpr int BPW = NB / NW;            // blocks per wave
  static_assert(NB % NW == 0 && BPW <= 4, "a wave's blocks must lie in one page");
  constexpr int HALF_TILE = 16384;        // K (or V^T) bytes per buffer
  constexpr int NBUF = 4;                 // LDS ring: tile j read, j+1 landed, j+2 and j+3 in flight
  constexpr int VBASE = NBUF * HALF_TILE; // V^T parts after the K parts of all buffers
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * NBUF * HALF_TILE];

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int tile_idx = block / a.n_kv_heads, g = block % a.n_kv_heads;
  const ExtendTile tile = a.tiles[tile_idx];
  const ExtendConvDesc cd = a.convs[tile.conv];
  const int prefix = cd.len - cd.q_len;
  const int q_hi = min(cd.q_len, tile.q0 + BM);
  const int pos_min = prefix + tile.q0, pos_max = prefix + q_hi - 1;
  const int n_kt = pos_max / kBN + 1;
  const int n_pg = (cd.len + kPageTokens - 1) / kPageTokens;
  const int32_t* pt = a.page_table + static_cast<size_t>(cd.slot) * a.max_pages;
  const int h = g * G + wave % G;
  const int qblk = wave / G;
  const int n_q_heads = a.n_kv_heads * G;
  const size_t head_stride = static_cast<size_t>(2 * kPageTokens * D);
  const size_t layer_base = static_cast<size_t>(a.layer) * a.n_pages * a.n_kv_heads * head_stride +
                            static_cast<size_t>(g) * head_stride;
  const size_t page_stride = static_cast<size_t>(a.n_kv_heads) * head_stride;
  const float c = a.scale_log2;
  const __attribute__((address_space(4))) int32_t* ptc =
      (const __attribute__((address_space(4))) int32_t*)reinterpret_cast<uintptr_t>(pt);

  // ---- copy side: block kb (1 KiB) of a tile = K rows 4kb .. 4kb+3 (page kb / 4) and V^T dims
  // 32 (kb % 4) .. +31 of page kb / 4; this wave copies blocks BPW*wave .. BPW*wave + BPW-1, all of
  // one page. The per-lane global offsets are fixed; only the page base changes per tile.
  const int q_w = (BPW * wave) / 4;
  uint32_t koff[BPW], voff[BPW];
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int quarter = (BPW * wave + i) % 4;
    const int row = 4 * quarter + lane / 16;                 // LDS row within the page
    const int chunk = (lane % 16) ^ row;                     // logical 16-byte chunk of that row
    // LDS row 8a + 4h + b holds key 8h + 4a + b (bits 2 and 3 swapped): the S^T accumulator
    // of lane half h then holds keys 8h .. 8h+7 of each 16-key step, the order of V^T in LDS.
    const int key = ((quarter & 1) << 3 | (quarter >> 1) << 2) + lane / 16;
    koff[i] = static_cast<uint32_t>(k_elem(key, chunk) * 2);
    const int dim = 32 * quarter + lane / 2;
    const int hv = (lane & 1) ^ ((dim >> 2) & 1) ^ ((dim >> 3) & 1);
    voff[i] = static_cast<uint32_t>(2 * kPageTokens * D + dim * 32 + hv * 16);
  }
  const uint32_t smem_base = lds_u32(smem);
  auto copy_tile = [&](int j, int buf) {
    const int lp = min(4 * j + q_w, n_pg - 1);
    const uint16_t* blk = a.pool + layer_base + static_cast<size_t>(ptc[lp]) * page_stride;
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int kb = BPW * wave + i;
      dma16(smem_base + buf * HALF_TILE + kb * 1024, blk, koff[i]);
      dma16(smem_base + VBASE + buf * HALF_TILE + kb * 1024, blk, voff[i]);
    }
  };

  // ---- read side: MFMA operand addresses (bytes within a buffer) -------------------------------
  // K operand of lane (col, half) for k-step ks: LDS row col (+32 kt2), logical chunk 2 ks + half,
  // stored at chunk (2 ks + half) ^ (row & 15). V^T operand for (kt2, j2, t): page 2 kt2 + j2,
  // dims 32 t + col, keys 8 half .. +7, stored in the block 4 (2 kt2 + j2) + t at col * 32 +
  // 16 (half ^ bit 2 of col ^ bit 3 of col).
  const int half = lane >> 5, col = lane & 31;
  uint32_t kaddr[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    kaddr[ks] = static_cast<uint32_t>(col * (2 * D) + (((2 * ks + half) ^ (col & 15)) * 16));
  const uint32_t vaddr =
      static_cast<uint32_t>(col * 32 + ((half ^ ((col >> 2) & 1) ^ ((col >> 3) & 1)) * 16));

  bf16x8 qop[KS];
  int qpos;
  {
    const int qi = tile.q0 + 32 * qblk + col;
    const bool valid = qi < cd.q_len;
    qpos = prefix + (valid ? qi : cd.q_len - 1);
    const uint16_t* qrow = a.q + (static_cast<size_t>(cd.q_row + (valid ? qi : 0)) * n_q_heads + h) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 x = ld16(qrow + 16 * ks + 8 * half);      // in bounds for padding rows too
      qop[ks] = as_bf16x8(valid ? x : make_uint4(0, 0, 0, 0));
    }
    // Q must have arrived before the loop: the compiler's own vector-memory waits then never
    // extend to the copies the loop keeps in flight (a wait at the loop head would drain them).
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" ::"v"(qop[ks]));
  }
  f32x16 o[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[t][e] = 0.f;
  float m_s = -INFINITY, l_run = 0.f;
  const bf16x2 ones = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};

  // Copies are issued for tiles past the end too (clamped to the last tile, whose pages past the
  // conversation's end are clamped to its last page), so every step issues the same number and
  // the counter waits below stay exact. Those keys are masked by the causal mask.
  copy_tile(0, 0);
  copy_tile(min(1, n_kt - 1), 1);
  copy_tile(min(2, n_kt - 1), 2);
  dma_wait_barrier<2 * BPW>();   // tiles 0 and 1 landed
  // K operands of the next tile are read into registers during the current tile's PV product.
  bf16x8 kop[KS][2];
  auto read_k = [&](int buf) {
    const uint8_t* kb = smem + buf * HALF_TILE;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
        kop[ks][kt2] = as_bf16x8(ld16(kb + kaddr[ks] + kt2 * 8192));
  };
  read_k(0);

  auto tile_step = [&](const int j, const int buf) {
    copy_tile(min(j + 3, n_kt - 1), (buf + 3) % NBUF);
    const uint8_t* vb = smem + VBASE + buf * HALF_TILE;
    f32x16 s[2];
#pragma unroll
    for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kt2][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
        s[kt2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[ks][kt2], qop[ks], s[kt2], 0, 0, 0);

    bf16x8 vop[2][2][DT];
#pragma unroll
    for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
      for (int j2 = 0; j2 < 2; ++j2)
#pragma unroll
        for (int t = 0; t < DT; ++t)
          vop[kt2][j2][t] = as_bf16x8(ld16(vb + vaddr + (4 * (2 * kt2 + j2) + t) * 1024));

    if (kBN * j + kBN - 1 > pos_min) {
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = kBN * j + 32 * kt2 + 16 * (e >> 3) + 8 * half + 4 * ((e >> 2) & 1) + (e & 3);
          if (key > qpos) s[kt2][e] = -INFINITY;
        }
    }
    // Weights against the running max m. If a lane's partial sum over its 32 keys of the tile
    // exceeds 2^8 or is not finite (always on the first tile, where m = -inf), the wave takes the
    // tile's row max, rescales O and l and recomputes the weights: every weight stays <= 2^8
    // without a max reduction on the common path.
    bf16x8 pop[2][2];
    auto weights = [&](float neg_m) {
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2) {
        float p[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) p[e] = fast_exp2(__builtin_fmaf(s[kt2][e], c, neg_m));
#pragma unroll
        for (int j2 = 0; j2 < 2; ++j2) {
          const uint4 pw = make_uint4(pack_bf16x2(p[8 * j2 + 0], p[8 * j2 + 1]),
                                      pack_bf16x2(p[8 * j2 + 2], p[8 * j2 + 3]),
                                      pack_bf16x2(p[8 * j2 + 4], p[8 * j2 + 5]),
                                      pack_bf16x2(p[8 * j2 + 6], p[8 * j2 + 7]));
          // the denominator sums the same bf16-rounded weights the PV product uses
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.x), ones, ps0, false);
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.y), ones, ps1, false);
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.z), ones, ps0, false);
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.w), ones, ps1, false);
          pop[kt2][j2] = __builtin_bit_cast(bf16x8, pw);
        }
      }
      return ps0 + ps1;
    };
    float ps = weights(-m_s);
    if (__builtin_amdgcn_ballot_w64(!(ps <= kSumLimit)) != 0) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt2][e]);
      const float m_new = fmaxf(m_s, halves_max(mx) * c);
      const float alpha = fast_exp2(m_s - m_new);
      m_s = m_new;
      l_run *= alpha;
#pragma unroll
      for (int t = 0; t < DT; ++t) o[t] *= alpha;
      ps = weights(-m_new);
    }
    l_run += ps;
#pragma unroll
    for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
      for (int j2 = 0; j2 < 2; ++j2)
#pragma unroll
        for (int t = 0; t < DT; ++t)
          o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[kt2][j2][t], pop[kt2][j2], o[t], 0, 0, 0);
    read_k((buf + 1) % NBUF);      // tile j+1 is in LDS (waited at the end of step j-1)
    // this wave's copies of tile j+2 have landed (those of tile j+3 may still fly); after the
    // barrier every wave's have.
    dma_wait_barrier<2 * BPW>();
  };
  for (int j = 0; j < n_kt; j += 4) {
    tile_step(j, 0);
    if (j + 1 < n_kt) tile_step(j + 1, 1);
    if (j + 2 < n_kt) tile_step(j + 2, 2);
    if (j + 3 < n_kt) tile_step(j + 3, 3);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no copy may land after the workgroup ends

  const int qi = tile.q0 + 32 * qblk + col;
  const float l_tot = halves_sum(l_run);
  if (qi < cd.q_len) {
    const float inv = 1.f / l_tot;
    uint16_t* orow = a.out + (static_cast<size_t>(cd.q_row + qi) * n_q_heads + h) * D;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int dim = 32 * t + 8 * e4 + 4 * half;
        st8(orow + dim, make_uint2(pack_bf16x2(o[t][4 * e4 + 0] * inv, o[t][4 * e4 + 1] * inv),
                                   pack_bf16x2(o[t][4 * e4 + 2] * inv, o[t][4 * e4 + 3] * inv)));
      }
  }
}

template <int G>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2)))
void attn_fwd_kernel(ExtendArgs a) {
  attn_fwd_block<G>(a, blockIdx.x);
}

// One layer of a mixed step in one launch (head_dim 128): the first n_ext workgroups are the
// extend tiles of the layer, the others each take one work item of the layer's decode split (8
// waves, as in the split kernel). Every workgroup gets the attention kernel's LDS ring and register
// budget (one per CU, two waves per SIMD); the decode split reads HBM as fast with two waves per
// SIMD as with three.
template <int G>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2)))
void mixed_layer_kernel(ExtendArgs ea, int n_ext, DecodeArgs da) {
  static_assert(kDecodeItemThreads == 512, "a decode work item fills one attention workgroup");
  __shared__ float xch[split_exchange_floats<128>()];
  if (static_cast<int>(blockIdx.x) < n_ext) {
    attn_fwd_block<G>(ea, blockIdx.x);
    return;
  }
  split_body<128>(da, blockIdx.x - n_ext, __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), xch);
}

// ------------------------------------------------------------------------------------------------
// head_dim 64: K/V staged through registers (global loads two tiles ahead, LDS stores of the next
// tile at the end of a step); V^T 4-key groups permuted in LDS to the accumulator's key order.
// ------------------------------------------------------------------------------------------------
template <int D, int G, int QT, int BM>
__global__ __launch_bounds__(64 * G * (BM / (32 * QT))) __attribute__((amdgpu_waves_per_eu(QT == 1 ? 2 : 1)))
void attn_fwd_staged_kernel(ExtendArgs a) {
  constexpr int NW = G * (BM / (32 * QT));  // waves: G query heads x BM/(32 QT) query blocks
  constexpr int NT = 64 * NW;          // threads
  constexpr int KS = D / 16;           // k-steps of QK^T (16 dims each)
  constexpr int DT = D / 32;           // 32-dim output tiles
  constexpr int CH = kBN * D / 8;      // 16-byte chunks per K (or V^T) tile
  constexpr int PER = CH / NT;         // chunks per thread per tile
  static_assert(CH % NT == 0, "tile chunks must divide the workgroup");
  __shared__ FwdSmem<D> sm;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int tile_idx = blockIdx.x / a.n_kv_heads, g = blockIdx.x % a.n_kv_heads;
  const ExtendTile tile = a.tiles[tile_idx];
  const ExtendConvDesc cd = a.convs[tile.conv];
  const int prefix = cd.len - cd.q_len;
  const int q_hi = min(cd.q_len, tile.q0 + BM);              // queries [q0, q_hi)
  const int pos_min = prefix + tile.q0, pos_max = prefix + q_hi - 1;
  const int n_kt = pos_max / kBN + 1;                        // key tiles 0 .. n_kt-1
  const int n_pg = (cd.len + kPageTokens - 1) / kPageTokens;
  const int32_t* pt = a.page_table + static_cast<size_t>(cd.slot) * a.max_pages;
  const int h = g * G + wave % G;                             // query head of this wave
  const int qblk = wave / G;                                  // query block (QT tiles of 32)
  const int n_q_heads = a.n_kv_heads * G;
  const size_t head_stride = static_cast<size_t>(2 * kPageTokens * D);
  const size_t layer_base = static_cast<size_t>(a.layer) * a.n_pages * a.n_kv_heads * head_stride +
                            static_cast<size_t>(g) * head_stride;
  const size_t page_stride = static_cast<size_t>(a.n_kv_heads) * head_stride;
  const float c = a.scale_log2;

  // ---- global -> register staging of one K/V tile (pages 4j .. 4j+3) ------------------------
  // Two register sets: the loads of tile j+2 are issued while tile j is computed and land in LDS
  // at the end of tile j+1, so each load has two tile-iterations to arrive.
  uint4 kregs[2][PER], vregs[2][PER];
  // A wave's 64 consecutive chunks always lie in one page, so the page id is wave-uniform and is
  // read with a scalar load: the vector-memory counter then only tracks K/V data, and waiting for
  // a page id never drains K/V loads still in flight for an earlier tile.
  const __attribute__((address_space(4))) int32_t* ptc =
      (const __attribute__((address_space(4))) int32_t*)reinterpret_cast<uintptr_t>(pt);
  auto load_tile = [&](int j, uint4 (&kreg)[PER], uint4 (&vreg)[PER]) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + u * NT;
      // Always load (pages past the end are clamped to the last page and zeroed when stored), so
      // the number of loads in flight is the same on every path and the waits stay precise.
      const int lp = min(__builtin_amdgcn_readfirstlane(4 * j + i / (2 * D)), n_pg - 1);
      const int w = i % (2 * D);
      const uint16_t* blk = a.pool + layer_base + static_cast<size_t>(ptc[lp]) * page_stride;
      kreg[u] = ld16(blk + w * 8);                          // K: sub-block w/64, key (w%64)/4
      vreg[u] = ld16(blk + kPageTokens * D + w * 8);        // V^T: dim w/2, keys 8*(w%2)..+8
    }
  };
  // LDS store of a staged tile. Only a tile that reaches past the end of the conversation needs
  // masking (uniform branch): K rows of pages past the end are zeroed and V of keys past the end
  // is zeroed, so no value read from a clamped page can reach the output.
  auto store_tile = [&](int buf, int j, const uint4 (&kreg)[PER], const uint4 (&vreg)[PER]) {
    const bool tail = kBN * (j + 1) > cd.len;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + u * NT;
      const int p = i / (2 * D), w = i % (2 * D);
      // K chunk w of the block: sub-block w / 64, key (w % 64) / 4, dims 32 (w / 64) + 8 (w % 4)
      const int row = kPageTokens * p + (w & 63) / 4, col8 = ((w >> 6) * 4 + (w & 3)) * 8;
      uint4 kx = kreg[u], vx = vreg[u];
      if (tail) {
        if (4 * j + p >= n_pg) kx = make_uint4(0, 0, 0, 0);
        const int key0 = kBN * j + kPageTokens * p + 8 * (w & 1);
        vx.x = mask_bf16x2(vx.x, key0 + 0 < cd.len, key0 + 1 < cd.len);
        vx.y = mask_bf16x2(vx.y, key0 + 2 < cd.len, key0 + 3 < cd.len);
        vx.z = mask_bf16x2(vx.z, key0 + 4 < cd.len, key0 + 5 < cd.len);
        vx.w = mask_bf16x2(vx.w, key0 + 6 < cd.len, key0 + 7 < cd.len);
      }
      st16(&sm.k[buf][row][col8], kx);
      const int dim = w >> 1, c0 = 2 * (w & 1);             // key groups c0, c0+1 of the page
      uint16_t* vrow = &sm.v[buf][dim][kPageTokens * p];
      st8(vrow + 4 * vt_group_pos(c0), make_uint2(vx.x, vx.y));
      st8(vrow + 4 * vt_group_pos(c0 + 1), make_uint2(vx.z, vx.w));
    }
  };

  // ---- Q operand in registers: query q0 + 32*(QT*qblk + qt) + lane%32, dims 16ks + 8*(lane/32)
  const int half = lane >> 5, col = lane & 31;
  bf16x8 qop[QT][KS];
  int qpos[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qi = tile.q0 + 32 * (QT * qblk + qt) + col;
    const bool valid = qi < cd.q_len;
    qpos[qt] = prefix + (valid ? qi : cd.q_len - 1);
    const uint16_t* qrow = a.q + (static_cast<size_t>(cd.q_row + (valid ? qi : 0)) * n_q_heads + h) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qop[qt][ks] = valid ? as_bf16x8(ld16(qrow + 16 * ks + 8 * half)) : bf16x8{};
  }

  f32x16 o[DT][QT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[t][qt][e] = 0.f;
  float m_s[QT], l_run[QT];   // running max (scaled, log2 units) and this lane's partial sum
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_s[qt] = -INFINITY;
    l_run[qt] = 0.f;
  }
  const bf16x2 ones = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};

  load_tile(0, kregs[0], vregs[0]);
  store_tile(0, 0, kregs[0], vregs[0]);
  load_tile(min(1, n_kt - 1), kregs[1], vregs[1]);
  __syncthreads();

  auto tile_step = [&](const int j, const int buf, uint4 (&kl)[PER], uint4 (&vl)[PER],
                       const uint4 (&ks_)[PER], const uint4 (&vs_)[PER]) {
    load_tile(min(j + 2, n_kt - 1), kl, vl);   // unconditional: same loads in flight on every path

    // S^T tiles (raw scores): [key subtile kt2][query tile qt]
    f32x16 s[2][QT];
#pragma unroll
    for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int e = 0; e < 16; ++e) s[kt2][qt][e] = 0.f;
    // All K operands of the tile are read from LDS before the first MFMA, so the LDS latency is
    // paid once per tile instead of once per MFMA.
    bf16x8 kop[KS][2];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
        kop[ks][kt2] = as_bf16x8(ld16(&sm.k[buf][32 * kt2 + col][16 * ks + 8 * half]));
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
        for (int qt = 0; qt < QT; ++qt)
          s[kt2][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[ks][kt2], qop[qt][ks], s[kt2][qt], 0, 0, 0);

    // V operands are read now: their LDS latency overlaps the softmax below.
    bf16x8 vop[2][2][DT];
#pragma unroll
    for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
      for (int j2 = 0; j2 < 2; ++j2)
#pragma unroll
        for (int t = 0; t < DT; ++t)
          vop[kt2][j2][t] = as_bf16x8(ld16(&sm.v[buf][32 * t + col][32 * kt2 + 16 * j2 + 8 * half]));

    // Online softmax, one query per lane and query tile; exp2 of c*s - m with c = log2(e)/sqrt(d).
    const bool need_mask = kBN * j + kBN - 1 > pos_min;
    bf16x8 pop[QT][2][2];  // [qt][kt2][j2]
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      if (need_mask) {
#pragma unroll
        for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = kBN * j + 32 * kt2 + 8 * (e >> 2) + 4 * half + (e & 3);
            if (key > qpos[qt]) s[kt2][qt][e] = -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt2][qt][e]);
      mx = halves_max(mx) * c;
      if (__builtin_amdgcn_ballot_w64(mx > m_s[qt] + kRescaleLog2) != 0) {
        const float m_new = fmaxf(m_s[qt], mx);
        const float alpha = fast_exp2(m_s[qt] - m_new);
        m_s[qt] = m_new;
        l_run[qt] *= alpha;
#pragma unroll
        for (int t = 0; t < DT; ++t) o[t][qt] *= alpha;
      }
      const float neg_m = -m_s[qt];
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int kt2 = 0; kt2 < 2; ++kt2) {
        float p[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) p[e] = fast_exp2(__builtin_fmaf(s[kt2][qt][e], c, neg_m));
#pragma unroll
        for (int j2 = 0; j2 < 2; ++j2) {
          const uint4 pw = make_uint4(pack_bf16x2(p[8 * j2 + 0], p[8 * j2 + 1]),
                                      pack_bf16x2(p[8 * j2 + 2], p[8 * j2 + 3]),
                                      pack_bf16x2(p[8 * j2 + 4], p[8 * j2 + 5]),
                                      pack_bf16x2(p[8 * j2 + 6], p[8 * j2 + 7]));
          // the denominator sums the same bf16-rounded weights the PV product uses
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.x), ones, ps0, false);
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.y), ones, ps1, false);
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.z), ones, ps0, false);
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pw.w), ones, ps1, false);
          pop[qt][kt2][j2] = __builtin_bit_cast(bf16x8, pw);
        }
      }
      l_run[qt] += ps0 + ps1;
    }

    // O^T += V^T . P^T over the 4 k-steps (16 keys each) of the tile.
#pragma unroll
    for (int kt2 = 0; kt2 < 2; ++kt2)
#pragma unroll
      for (int j2 = 0; j2 < 2; ++j2)
#pragma unroll
        for (int t = 0; t < DT; ++t)
#pragma unroll
          for (int qt = 0; qt < QT; ++qt)
            o[t][qt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[kt2][j2][t], pop[qt][kt2][j2], o[t][qt], 0, 0, 0);

    // Unconditional: past the last tile it stores a masked tile that is never read (the buffer's
    // previous tile was consumed before the last barrier), and the store needs no branch.
    store_tile(buf ^ 1, j + 1, ks_, vs_);
    __syncthreads();
  };
  for (int j = 0; j < n_kt; j += 2) {
    tile_step(j, 0, kregs[0], vregs[0], kregs[1], vregs[1]);
    if (j + 1 < n_kt) tile_step(j + 1, 1, kregs[1], vregs[1], kregs[0], vregs[0]);
  }

  // Normalise and write: lane owns query col of tile qt, dims 32t + 8(e/4) + 4*half + e%4.
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int qi = tile.q0 + 32 * (QT * qblk + qt) + col;
    const float l_tot = halves_sum(l_run[qt]);
    if (qi >= cd.q_len) continue;
    const float inv = 1.f / l_tot;
    uint16_t* orow = a.out + (static_cast<size_t>(cd.q_row + qi) * n_q_heads + h) * D;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int dim = 32 * t + 8 * e4 + 4 * half;
        st8(orow + dim, make_uint2(pack_bf16x2(o[t][qt][4 * e4 + 0] * inv, o[t][qt][4 * e4 + 1] * inv),
                                   pack_bf16x2(o[t][qt][4 * e4 + 2] * inv, o[t][qt][4 * e4 + 3] * inv)));
      }
  }
}

// head_dim 128: 32 queries per wave, eight waves (two per SIMD); head_dim 64: 64 queries
// per wave, G waves.
template <int D, int G>
static void launch_fwd(const ExtendArgs& a, int n_tiles, int n_kv_heads, hipStream_t stream) {
  if constexpr (D == 128) {
    attn_fwd_kernel<G><<<n_tiles * n_kv_heads, 512, 0, stream>>>(a);
  } else {
    attn_fwd_staged_kernel<D, G, 2, kBM><<<n_tiles * n_kv_heads, 64 * G * (kBM / 64), 0, stream>>>(a);
  }
}

int extend_query_tile(int head_dim, int group) { return head_dim == 128 ? 256 / group : kBM; }

static ExtendArgs make_extend_args(const PoolGeom& g, int layer, const ExtendConvDesc* d_convs,
                                   const ExtendTile* d_tiles, const void* q, void* out) {
  ExtendArgs a;
  a.pool = static_cast<const uint16_t*>(g.pool);
  a.n_pages = g.n_pages;
  a.n_kv_heads = g.n_kv_heads;
  a.layer = layer;
  a.page_table = g.page_table;
  a.max_pages = g.max_pages;
  a.convs = d_convs;
  a.tiles = d_tiles;
  a.q = static_cast<const uint16_t*>(q);
  a.out = static_cast<uint16_t*>(out);
  a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(static_cast<double>(g.head_dim)));
  return a;
}

hipError_t launch_extend(const PoolGeom& g, int layer, const ExtendConvDesc* d_convs,
                         const ExtendTile* d_tiles, int n_tiles, const void* q, void* out,
                         hipStream_t stream) {
  if (n_tiles == 0) return hipSuccess;
  const ExtendArgs a = make_extend_args(g, layer, d_convs, d_tiles, q, out);
  const int G = g.n_q_heads / g.n_kv_heads;
#define CS_FWD_CASE(DD, GG)                                   \
  if (g.head_dim == DD && G == GG) {                          \
    launch_fwd<DD, GG>(a, n_tiles, g.n_kv_heads, stream);     \
    return hipGetLastError();                                 \
  }
  CS_FWD_CASE(128, 1) CS_FWD_CASE(128, 2) CS_FWD_CASE(128, 4) CS_FWD_CASE(128, 8)
  CS_FWD_CASE(64, 1) CS_FWD_CASE(64, 2) CS_FWD_CASE(64, 4) CS_FWD_CASE(64, 8)
#undef CS_FWD_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_mixed_layer(const PoolGeom& g, int layer, const ExtendConvDesc* d_ext_convs,
                              const ExtendTile* d_tiles, int n_tiles, const void* q_ext,
                              void* out_ext, const DecodeConvDesc* d_dec_convs,
                              const int32_t* d_dec_order, int n_dec_convs, int n_items, int split_tokens,
                              const void* q_dec, float* partials, void* direct_out, hipStream_t stream) {
  if (g.head_dim != 128 || n_tiles == 0 || n_dec_convs == 0) return hipErrorInvalidValue;
  if (d_dec_order == nullptr || n_items < n_dec_convs) return hipErrorInvalidValue;
  if (direct_out != nullptr && n_items != n_dec_convs) return hipErrorInvalidValue;
  const ExtendArgs ea = make_extend_args(g, layer, d_ext_convs, d_tiles, q_ext, out_ext);
  DecodeArgs da = make_decode_args(g, layer, d_dec_convs, d_dec_order, n_dec_convs, n_items, split_tokens,
                                   q_dec, direct_out, partials);
  da.direct = direct_out != nullptr;
  const int n_ext = n_tiles * g.n_kv_heads;
  const int blocks = n_ext + n_items * g.n_kv_heads;
  switch (g.n_q_heads / g.n_kv_heads) {
    case 1: mixed_layer_kernel<1><<<blocks, 512, 0, stream>>>(ea, n_ext, da); break;
    case 2: mixed_layer_kernel<2><<<blocks, 512, 0, stream>>>(ea, n_ext, da); break;
    case 4: mixed_layer_kernel<4><<<blocks, 512, 0, stream>>>(ea, n_ext, da); break;
    case 8: mixed_layer_kernel<8><<<blocks, 512, 0, stream>>>(ea, n_ext, da); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace cs
