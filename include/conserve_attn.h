/*
 * conserve_attn.h -- C ABI of the paged-KV attention hot path under conversation-level
 * disaggregated serving (arxiv 2606.01839, "Observation, Not Prediction").
 *
 * The paper (Section 4 and Fig. 9) binds each agentic conversation to one decoder for its whole
 * life: the turn-1 prompt is prefilled (on the prefiller), the resulting KV cache is transferred
 * exactly once, and the first decode plus every later turn's incremental prefill ("append") and
 * decode run on the decoder against the conversation's ever-growing KV cache (Section 1; Section
 * 3.1 "prefix caching" and "KV cache transfer"; Section 3.2 "memory-bound" decode). This library is
 * the data-parallel part of that: a pool of 16-token KV pages per GPU, conversations that own pages,
 * and the kernels that append KV, attend (turn-1 prefill, extend, batched decode) and move a
 * conversation's KV out of / into a pool (the one-time transfer).
 *
 * Conventions for every call
 * --------------------------
 *  - Device pointers: every `void*` named k, v, q, out, dst, src, kv_base, ws_base is a device
 *    address on the current HIP device; the caller owns that memory and keeps it alive until the
 *    stream reaches the call. Host pointers: cs_conv arrays, q_lens, and the out-parameters.
 *  - Element type: bf16 (IEEE binary32 with the low 16 bits dropped) everywhere; accumulation fp32.
 *  - Append-then-attend: cs_kv_append is the only writer of a conversation's K/V. Attention calls
 *    take queries for the LAST q_len positions of each conversation; query i of a conversation of
 *    length L sits at position p = L - q_len + i and sees keys 0..p (itself included). Softmax
 *    scale is exactly 1/sqrt(head_dim). Query head h reads KV head h / (n_q_heads / n_kv_heads).
 *  - Errors: every call validates all arguments before changing any state; on error it returns a
 *    negative cs_status, changes nothing, and sets a thread-local message (cs_last_error). Nothing
 *    aborts or throws across this ABI. CS_EHIP reports a failing HIP runtime call; an append that
 *    fails so still changes no length and no page (its reserved pages return to the free list);
 *    cs_mixed_step's append is complete when a later attention launch fails; after any CS_EHIP
 *    the outputs of the failing call are undefined.
 *  - Asynchrony: host metadata (lengths, page tables) is committed when the call returns; kernels
 *    and the small metadata uploads they need are enqueued on `stream` (a hipStream_t, 0 = null
 *    stream). No call synchronises the device, except that switching a pool to another stream
 *    makes the new stream wait (hipStreamWaitEvent) for work already enqueued on the previous one.
 *  - A pool is not thread-safe: one host thread at a time.
 */
#ifndef CONSERVE_ATTN_H
#define CONSERVE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct cs_pool cs_pool;   /* opaque; library-owned host metadata */
typedef int32_t cs_conv;          /* conversation handle (>= 0) */
typedef void* cs_stream;          /* hipStream_t */
typedef int32_t cs_status;

enum {
  CS_OK = 0,
  CS_EINVAL = -1,  /* bad argument: null pointer, bad size, duplicate conversation, wire mismatch */
  CS_ENOMEM = -2,  /* pool has too few free pages / no free conversation slot / ring too small */
  CS_ENOENT = -3,  /* unknown or destroyed conversation handle */
  CS_ESTATE = -4,  /* call not valid in the conversation's state (e.g. q_len > length) */
  CS_ERANGE = -5,  /* index out of range (layer, page capacity of a conversation) */
  CS_EHIP = -6,    /* a HIP runtime call failed */
  CS_EBUSY = -7    /* placement refused: the prefiller is saturated (conserve_sched.h) */
};

#define CS_PAGE_TOKENS 16

typedef struct {
  int32_t n_layers;            /* >= 1 */
  int32_t n_q_heads;           /* multiple of n_kv_heads; n_q_heads/n_kv_heads in {1,2,4,8} */
  int32_t n_kv_heads;          /* >= 1 */
  int32_t head_dim;            /* 64 or 128 */
  int32_t max_convs;           /* live conversations at once, 1 .. 2^20 */
  int32_t max_pages_per_conv;  /* longest conversation, in 16-token pages */
  int64_t n_pages;             /* pool capacity in pages; a page holds 16 tokens of every layer */
} cs_pool_desc;

/*
 * KV pool layout (device, caller-allocated, cs_pool_kv_bytes(desc) bytes, 256-byte aligned):
 *   pool[layer][page][kv_head] = one 4*16*head_dim-byte block:
 *     K part: head_dim/32 sub-blocks, sub-block s = K[16 tokens][dims 32s .. 32s+31] token-major
 *             (each sub-block 1 KiB: what one matrix-core operand load of 16 keys reads), then
 *     V^T[head_dim][16] dimension-major (each row holds one dimension of the page's 16 tokens).
 * Token slots >= length in a conversation's last page always hold zeros (append and unpack write
 * them), so a page is never read past the conversation's end with undefined contents.
 */
size_t cs_pool_kv_bytes(const cs_pool_desc* desc);

/* Device workspace bytes the pool needs (page-table mirror, decode partials, metadata ring). */
size_t cs_pool_workspace_bytes(const cs_pool_desc* desc);

/*
 * Create a pool over caller memory. Physical pages are handed out from a free list shuffled by
 * `placement_seed`, so page placement is random (results never depend on it). Pinned host staging
 * memory for metadata uploads is allocated by the pool's first device call (an append, unpack or
 * attention call) and freed by cs_pool_destroy.
 * Errors: CS_EINVAL (bad descriptor, null/short/misaligned buffers), CS_EHIP.
 */
cs_status cs_pool_create(const cs_pool_desc* desc, void* kv_base, size_t kv_bytes, void* ws_base,
                         size_t ws_bytes, uint64_t placement_seed, cs_pool** out);

/* Destroy host state; never frees caller memory. Waits for the pool's enqueued work first. */
cs_status cs_pool_destroy(cs_pool* pool);

/* Pages held by live conversations and pages still free (the decoder's active KV occupancy that
 * the paper's reactive scheduler reads, Section 4.2; freed when a conversation ends). */
cs_status cs_pool_occupancy(const cs_pool* pool, int64_t* used_pages, int64_t* free_pages);

/* New empty conversation (Section 4.2: a conversation enters at its first turn).
 * Errors: CS_EINVAL (null out), CS_ENOMEM (max_convs live). */
cs_status cs_conv_create(cs_pool* pool, cs_conv* out);

/* End a conversation and return its pages to the pool (Section 4.2: occupancy is decremented at
 * termination). The caller must not destroy a conversation that enqueued work still reads.
 * Errors: CS_ENOENT. */
cs_status cs_conv_destroy(cs_pool* pool, cs_conv conv);

/* Current length in tokens. Errors: CS_ENOENT, CS_EINVAL. */
cs_status cs_conv_len(const cs_pool* pool, cs_conv conv, int64_t* tokens);

/* Copy the conversation's physical page ids (logical order) into out[0..cap); *n = page count.
 * Errors: CS_ENOENT, CS_EINVAL (null), CS_ERANGE (cap < page count; *n still set). */
cs_status cs_conv_pages(const cs_pool* pool, cs_conv conv, int32_t* out, int64_t cap, int64_t* n);

/*
 * Append n_new tokens of K and V for every layer (Section 2.1: decode appends one KV entry per
 * generated token; Section 3.1: a later turn adds the entries of its appended tokens).
 * k, v: device, [n_layers][n_new][n_kv_heads][head_dim] bf16, contiguous.
 * Reserves ceil((len+n_new)/16) - ceil(len/16) new pages first; on CS_ENOMEM nothing changes.
 * n_new == 0 is a no-op. Errors: CS_ENOENT, CS_EINVAL, CS_ENOMEM, CS_ERANGE, CS_EHIP.
 */
cs_status cs_kv_append(cs_pool* pool, cs_conv conv, int32_t n_new, const void* k, const void* v,
                       cs_stream stream);

/*
 * Batched append: conversation convs[i] receives n_new[i] tokens; k, v are
 * [n_layers][sum(n_new)][n_kv_heads][head_dim] with the conversations' tokens concatenated in
 * batch order. All-or-nothing page reservation. Conversations must be distinct.
 */
cs_status cs_kv_append_batch(cs_pool* pool, int32_t n_convs, const cs_conv* convs,
                             const int32_t* n_new, const void* k, const void* v, cs_stream stream);

/*
 * Turn-1 causal prefill (Section 3.1: the compute-bound first-turn prefill). For each conversation
 * q_lens[i] must equal its length (its whole content is the prompt just appended).
 * q:   device [sum(q_lens)][n_q_heads][head_dim] bf16, conversations in batch order.
 * out: device, same shape; bf16 (round to nearest even) of softmax(q k^T / sqrt(d)) v, causal.
 * Errors: CS_EINVAL (null, duplicate conv, q_len < 0), CS_ENOENT, CS_ESTATE (q_len != length),
 * CS_ERANGE (layer), CS_ENOMEM (metadata larger than the ring), CS_EHIP.
 */
cs_status cs_attn_prefill_turn1(cs_pool* pool, int32_t n_convs, const cs_conv* convs,
                                const int32_t* q_lens, int32_t layer, const void* q, void* out,
                                cs_stream stream);

/*
 * Extend-prefill of a later turn (Section 3.1 "prefix caching": the appended tokens attend to the
 * whole cached history and causally among themselves; Section 4: it runs on the pinned decoder).
 * Same arguments as cs_attn_prefill_turn1 but 0 <= q_lens[i] <= length (q_len == length is a full
 * prefill, q_len == 1 a decode). Errors as above, CS_ESTATE when q_len > length.
 */
cs_status cs_attn_extend(cs_pool* pool, int32_t n_convs, const cs_conv* convs,
                         const int32_t* q_lens, int32_t layer, const void* q, void* out,
                         cs_stream stream);

/*
 * Batched single-token decode (Section 2.1 / 3.2: each step reads the whole cache of every
 * conversation in the batch; memory-bound). The query of convs[i] is its last position.
 * q, out: device [n_convs][n_q_heads][head_dim] bf16. Conversations distinct, length >= 1.
 * Split-K over fixed logical token ranges plus a fixed-order log-sum-exp merge: the result is
 * bitwise deterministic and independent of physical page placement.
 * Errors: CS_EINVAL, CS_ENOENT, CS_ESTATE (length 0), CS_ERANGE, CS_ENOMEM, CS_EHIP.
 */
cs_status cs_attn_decode_batch(cs_pool* pool, int32_t n_convs, const cs_conv* convs,
                               int32_t layer, const void* q, void* out, cs_stream stream);

/*
 * Allocation-free variant of cs_attn_decode_batch, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc). Same
 * arguments, semantics and output bits as cs_attn_decode_batch; the only difference is where the
 * decode split keeps its partial records: in a static device array of the library (16 MiB =
 * 4,194,304 floats on each GPU, held until the process ends) instead of the pool's workspace.
 * The call allocates no device or pinned memory and creates no HIP objects (the device address of
 * the array is looked up once per device); host-side planning uses the C++ heap. It launches
 * untimed: cs_profile_* does not see it.
 * Every call on one GPU shares that GPU's array: calls that overlap on one GPU (on different
 * streams, or from different pools on different host threads) race and must not be issued.
 * Errors: as cs_attn_decode_batch; CS_ENOMEM when the batch's partial records
 * (n_items * n_q_heads * (head_dim + 4) floats; batches whose conversations are each one work item
 * need none) exceed the array; CS_ESTATE when the pool has made no device call yet (its first one
 * allocates its metadata ring; an append or unpack that filled it always has); CS_EINVAL when the
 * current device is not the pool's.
 */
cs_status cs_attn_decode_batch_noalloc(cs_pool* pool, int32_t n_convs, const cs_conv* convs,
                                       int32_t layer, const void* q, void* out, cs_stream stream);

/*
 * One step of a decoder serving agentic conversations (Section 4: after the one-time transfer a
 * conversation's later turns -- incremental prefill of appended tokens and decoding -- run on its
 * decoder; Section 2.1: dynamic batching lets requests join and leave every iteration). In one
 * call: conversations ext_convs[i] append an extend chunk of ext_lens[i] >= 1 tokens and
 * conversations dec_convs[j] append one decoded token (all layers), then for every layer the extend
 * queries attend (as cs_attn_extend) and the decode queries attend (as cs_attn_decode_batch).
 * All conversations must be distinct.
 *   k, v:     [n_layers][sum(ext_lens) + n_dec][n_kv_heads][head_dim], extend tokens first
 *   q_ext:    [n_layers][sum(ext_lens)][n_q_heads][head_dim];  out_ext same shape
 *   q_dec:    [n_layers][n_dec][n_q_heads][head_dim];          out_dec same shape
 * The batch metadata is uploaded once and reused by every layer's launches. When both parts are
 * present, the extend launches run on a second stream owned by the pool, forked from `stream`
 * after the append and joined back into it before the call returns: work enqueued on `stream`
 * afterwards (and a synchronisation of `stream`) sees every output of the step.
 * flags = 0: every layer's queries are inputs of the call, so no layer waits for another; the
 *   extend work of all layers overlaps the decode work of all layers, and the decode merge of
 *   layer l-1 shares one launch with the decode split of layer l (two partial buffers alternate).
 * flags = CS_MIXED_LAYER_ORDERED: the order of a model forward pass, where layer l+1's queries
 *   depend on layer l's output: layer l's extend and decode overlap each other, and layer l+1
 *   starts only when both are complete. At head_dim 128 with both parts present, a layer is one
 *   launch holding its extend tiles and its decode split, then the decode merge; otherwise the
 *   layer's extend runs on the second stream beside its decode.
 * Outputs are bitwise the same either way (and the same as the separate calls).
 * Errors: as cs_kv_append_batch, cs_attn_extend and cs_attn_decode_batch; CS_EINVAL for unknown
 * flags.
 */
enum { CS_MIXED_LAYER_ORDERED = 1 };
cs_status cs_mixed_step(cs_pool* pool, int32_t n_ext, const cs_conv* ext_convs,
                        const int32_t* ext_lens, int32_t n_dec, const cs_conv* dec_convs,
                        const void* k, const void* v, const void* q_ext, void* out_ext,
                        const void* q_dec, void* out_dec, uint32_t flags, cs_stream stream);

/*
 * Version of the transfer wire format of cs_kv_pack / cs_kv_unpack below. The format is frozen at
 * this version: it is the pool's block format as of version 1, and a later change of the pool's
 * private block layout keeps pack and unpack reading and writing exactly this format (a new format
 * would take a new version number).
 */
#define CS_WIRE_FORMAT_VERSION 1

/* Wire size of a conversation's KV: n_layers * ceil(len/16) * n_kv_heads * 64 * head_dim bytes. */
cs_status cs_kv_pack_size(const cs_pool* pool, cs_conv conv, size_t* bytes);

/*
 * Gather a conversation's pages in logical order into a contiguous wire buffer (the sending half
 * of the one-time turn-1 KV transfer, Section 4 and Section 3.1 "KV cache transfer").
 * Wire layout: [layer][logical page][kv_head] blocks in the pool's block format (K part in
 * 32-dim token-major sub-blocks, then V^T[d][16]); token slots >= length are written as zeros. dst: device, dst_bytes must equal
 * cs_kv_pack_size. Errors: CS_ENOENT, CS_EINVAL, CS_EHIP.
 */
cs_status cs_kv_pack(const cs_pool* pool, cs_conv conv, void* dst, size_t dst_bytes,
                     cs_stream stream);

/*
 * Receiving half of the transfer: create a conversation of n_tokens tokens in `pool`, take fresh
 * pages from its (randomly placed) free list and scatter the wire buffer into them. src_bytes must
 * equal the wire size for n_tokens with this pool's shape; tail slots are written as zeros.
 * Errors: CS_EINVAL (size mismatch, n_tokens < 1), CS_ENOMEM, CS_ERANGE, CS_EHIP.
 */
cs_status cs_kv_unpack(cs_pool* pool, const void* src, size_t src_bytes, int64_t n_tokens,
                       cs_conv* out_conv, cs_stream stream);

/*
 * Instrumentation (per-kernel timing; not part of the attention path). Between cs_profile_start
 * and cs_profile_stop every kernel the pool launches is bracketed by two HIP timing events on its
 * stream, except in cs_mixed_step, where one pair of events brackets the extend launches of all
 * layers and one pair the decode launches of all layers but the final merge (their time then
 * includes the gaps between those launches). cs_profile_stop waits for the events, writes the
 * summed milliseconds and the launch count per kernel kind into ms[CS_PROF_KINDS] and
 * launches[CS_PROF_KINDS], and disables timing.
 * Errors: CS_EINVAL (null), CS_EHIP.
 */
enum {
  CS_PROF_APPEND = 0,        /* kv append kernel */
  CS_PROF_PACK = 1,          /* kv pack kernel */
  CS_PROF_UNPACK = 2,        /* kv unpack kernel */
  CS_PROF_DECODE_SPLIT = 3,  /* decode split-K kernel */
  CS_PROF_DECODE_MERGE = 4,  /* decode merge kernel */
  CS_PROF_ATTN_FWD = 5,      /* prefill / extend attention kernel */
  CS_PROF_MIXED_LAYER = 6,   /* one layer's extend tiles + decode split in one launch */
  CS_PROF_KINDS = 7
};
cs_status cs_profile_start(cs_pool* pool);
cs_status cs_profile_stop(cs_pool* pool, double* ms, int64_t* launches);

/*
 * Instrumentation: properties of a HIP device that measurements are logged with (from
 * hipGetDeviceProperties). Errors: CS_EINVAL (null), CS_EHIP (no such device).
 */
typedef struct {
  char name[256];
  char arch[64];                 /* gcnArchName, e.g. "gfx950:sramecc+:xnack-" */
  int32_t cu_count;              /* compute units */
  int32_t clock_khz;             /* peak engine clock */
  int32_t memory_clock_khz;      /* peak memory clock */
  int32_t memory_bus_width_bits;
  int64_t lds_per_cu_bytes;      /* shared memory per compute unit */
  int64_t lds_per_block_bytes;   /* shared memory one workgroup may use */
  int64_t l2_bytes;              /* L2 cache size the runtime reports */
  int64_t total_mem_bytes;
} cs_device_info_t;
cs_status cs_device_info(int32_t device, cs_device_info_t* out);

/*
 * Instrumentation: read `bytes` (a multiple of 16) of device memory at `src` once with the
 * non-temporal 16-byte loads the decode and pack kernels use, on 8 workgroups per compute unit of
 * the current device, enqueued on `stream`; `sink` is 4 bytes of device memory that the kernel
 * writes only if the XOR of everything read equals 0x9E3779B9 (it exists so the loads stay live).
 * Time it with events on `stream` to get what streaming reads reach on the part.
 * Errors: CS_EINVAL (null pointers, bytes not a multiple of 16), CS_EHIP.
 */
cs_status cs_probe_stream_read(const void* src, size_t bytes, void* sink, cs_stream stream);

/*
 * Test instrumentation of the error paths: after `after` more kernel launches of this pool
 * succeed, every later launch of the pool reports CS_EHIP ("failure injected") without launching
 * anything, until the call is made again with after < 0 (off, the default). The failing call
 * behaves as on a real HIP launch failure at that point. Errors: CS_EINVAL (null pool).
 */
cs_status cs_debug_fail_launches(cs_pool* pool, int64_t after);

/* Message of the last failing call on this thread ("" if none). Valid until the next call. */
const char* cs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CONSERVE_ATTN_H */
