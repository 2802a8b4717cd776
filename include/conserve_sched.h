/*
 * conserve_sched.h -- conversation-level placement over the KV page pools of conserve_attn.h:
 * the reactive scheduler and the decoder provisioning rule of arxiv 2606.01839 ("Observation, Not
 * Prediction"), Section 4.
 *
 * The paper places a conversation once, from two observable signals (Section 4.2): the prefill
 * latency curve, profiled offline as a deterministic function of the turn-1 input length (Section
 * 3.1 finds it quadratic), and each decoder's active KV-cache occupancy, which drops when a
 * conversation ends. Every turn-1 prefill goes to the prefiller; after the one-time KV transfer
 * the conversation is bound, for its whole life, to the decoder with the lowest occupancy. When
 * the prefiller or the decoders are saturated the *next* conversation is routed elsewhere; nothing
 * already placed moves. Section 4.1 sizes the decoder tier from the prefiller's saturation rate.
 *
 * Host-only calls (no device work, no allocation on the device); conventions as in
 * conserve_attn.h: validation before any state change, negative cs_status plus cs_last_error()
 * on error, nothing aborts. A scheduler is not thread-safe.
 */
#ifndef CONSERVE_SCHED_H
#define CONSERVE_SCHED_H

#include "conserve_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Prefill latency curve t(L) = c0 + c1 L + c2 L^2 seconds for a turn-1 input of L tokens. */
typedef struct {
  double c0, c1, c2;
} cs_prefill_curve;

/*
 * Least-squares fit of the curve to n measured (tokens[i], seconds[i]) samples (Section 3.1:
 * prefill latency grows quadratically with input length). Needs n >= 3 with at least three
 * distinct lengths and finite times. *r2 (may be null) = 1 - SS_res / SS_tot.
 * Errors: CS_EINVAL (null, too few or degenerate samples).
 */
cs_status cs_prefill_curve_fit(int32_t n, const int64_t* tokens, const double* seconds,
                               cs_prefill_curve* out, double* r2);

/* Expected prefill seconds of a tokens-long prompt. Errors: CS_EINVAL (null). */
cs_status cs_prefill_curve_eval(const cs_prefill_curve* curve, int64_t tokens, double* seconds);

/*
 * Decoder provisioning (Section 4.1). With prefill throughput T_p (input tokens/s) and mean
 * turn-1 length L_in the prefiller saturates at R* = T_p / L_in conversations/s. N decoders of
 * throughput T_d (tokens/s), each holding B conversations, serve conversations that bring L_d
 * decoder-side tokens and live W seconds when N T_d >= R* L_d and N B >= R* W. Outputs (any may be
 * null): R*, the two bounds R* L_d / T_d and R* W / B, and N = the smallest integer greater than
 * both. Errors: CS_EINVAL (an input <= 0 or not finite, N beyond int32).
 */
cs_status cs_provision_decoders(double prefill_tokens_per_s, double mean_turn1_tokens,
                                double decoder_tokens_per_s, double mean_decoder_tokens,
                                double convs_per_decoder, double mean_lifetime_s,
                                double* saturation_rate, double* n_throughput, double* n_memory,
                                int32_t* n_decoders);

/*
 * Binding rule on explicit occupancies (Section 4.2): the decoder i with free_pages[i] >=
 * need_pages and the lowest used_pages[i] / (used_pages[i] + free_pages[i]) (exact comparison;
 * ties to the lower index). *decoder = -1 and CS_ENOMEM when none can hold the conversation.
 * Errors: CS_EINVAL (null, n < 1, negative counts).
 */
cs_status cs_place_least_occupied(int32_t n, const int64_t* used_pages, const int64_t* free_pages,
                                  int64_t need_pages, int32_t* decoder);

typedef struct cs_sched cs_sched;  /* opaque */

/*
 * Scheduler over n_decoders decoder pools (created by the caller with conserve_attn.h; the
 * scheduler only reads their occupancy and never owns them). max_wait_s bounds the expected wait
 * of a new conversation's turn-1 prefill behind the prefiller's admitted work. n_decoders = 0
 * (decoders may then be null) makes an admission-only scheduler, for callers that keep decoder
 * occupancy themselves and bind with cs_place_least_occupied (e.g. a host simulation);
 * cs_sched_bind on it fails with CS_EINVAL.
 * Errors: CS_EINVAL (null curve/out, null pools with n_decoders > 0, n_decoders < 0, max_wait_s
 * < 0 or not finite).
 */
cs_status cs_sched_create(const cs_prefill_curve* curve, double max_wait_s, int32_t n_decoders,
                          cs_pool* const* decoders, cs_sched** out);
cs_status cs_sched_destroy(cs_sched* sched);

/*
 * Admission of a new conversation at its first turn, arriving at now_s (seconds, caller's clock,
 * non-decreasing across calls). Its turn-1 prefill queues on the prefiller behind the admitted
 * work: it starts at max(now_s, busy_until) and takes curve(turn1_tokens) seconds; *start_s and
 * *done_s (may be null) receive both. CS_EBUSY, with nothing changed, when the expected wait
 * max(0, busy_until - now_s) exceeds max_wait_s: route the conversation elsewhere.
 * Errors: CS_EINVAL (null sched, turn1_tokens < 1, now_s not finite), CS_EBUSY.
 */
cs_status cs_sched_admit(cs_sched* sched, int64_t turn1_tokens, double now_s, double* start_s,
                         double* done_s);

/*
 * Bind a conversation whose KV cache holds kv_tokens tokens (after its turn-1 prefill, before the
 * transfer) to a decoder: cs_place_least_occupied over the decoders' cs_pool_occupancy with
 * need_pages = ceil(kv_tokens / 16). The caller then unpacks the transferred KV into
 * decoders[*decoder] (cs_kv_unpack), which raises that pool's occupancy; ending the conversation
 * (cs_conv_destroy) lowers it again.
 * Errors: CS_EINVAL (null, kv_tokens < 1), CS_ENOMEM (*decoder = -1: every decoder is too full).
 */
cs_status cs_sched_bind(cs_sched* sched, int64_t kv_tokens, int32_t* decoder);

#ifdef __cplusplus
}
#endif

#endif /* CONSERVE_SCHED_H */
