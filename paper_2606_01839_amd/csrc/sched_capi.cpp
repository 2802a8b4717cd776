// C ABI of the placement layer (declared in include/conserve_sched.h): validation and the pools'
// occupancy around the host-only scheduler of host/sched.{hpp,cpp}.
#include "conserve_sched.h"

#include <cmath>
#include <new>
#include <vector>

#include "host/host_state.hpp"
#include "host/sched.hpp"

namespace cs {
cs_status api_fail(cs_status code, const char* msg);  // capi.cpp: sets cs_last_error()
}  // namespace cs

struct cs_sched {
  cs::Admission admission;
  std::vector<cs_pool*> decoders;
  cs_sched(const cs::PrefillCurve& c, double max_wait) : admission(c, max_wait) {}
};

extern "C" {

cs_status cs_prefill_curve_fit(int32_t n, const int64_t* tokens, const double* seconds,
                               cs_prefill_curve* out, double* r2) {
  if (!tokens || !seconds || !out) return cs::api_fail(CS_EINVAL, "null argument");
  cs::PrefillCurve c;
  if (!cs::fit_prefill_curve(tokens, seconds, n, &c, r2))
    return cs::api_fail(CS_EINVAL, "need >= 3 finite samples with at least three distinct lengths");
  out->c0 = c.c0;
  out->c1 = c.c1;
  out->c2 = c.c2;
  return CS_OK;
}

cs_status cs_prefill_curve_eval(const cs_prefill_curve* curve, int64_t tokens, double* seconds) {
  if (!curve || !seconds) return cs::api_fail(CS_EINVAL, "null argument");
  cs::PrefillCurve c;
  c.c0 = curve->c0;
  c.c1 = curve->c1;
  c.c2 = curve->c2;
  *seconds = c.eval(tokens);
  return CS_OK;
}

cs_status cs_provision_decoders(double prefill_tokens_per_s, double mean_turn1_tokens,
                                double decoder_tokens_per_s, double mean_decoder_tokens,
                                double convs_per_decoder, double mean_lifetime_s,
                                double* saturation_rate, double* n_throughput, double* n_memory,
                                int32_t* n_decoders) {
  cs::Provisioning p;
  if (!cs::provision_decoders(prefill_tokens_per_s, mean_turn1_tokens, decoder_tokens_per_s,
                              mean_decoder_tokens, convs_per_decoder, mean_lifetime_s, &p))
    return cs::api_fail(CS_EINVAL, "provisioning inputs must be positive and finite (N <= int32)");
  if (saturation_rate) *saturation_rate = p.saturation_rate;
  if (n_throughput) *n_throughput = p.n_throughput;
  if (n_memory) *n_memory = p.n_memory;
  if (n_decoders) *n_decoders = p.n_decoders;
  return CS_OK;
}

cs_status cs_place_least_occupied(int32_t n, const int64_t* used_pages, const int64_t* free_pages,
                                  int64_t need_pages, int32_t* decoder) {
  if (!used_pages || !free_pages || !decoder || n < 1)
    return cs::api_fail(CS_EINVAL, "null argument or n < 1");
  if (need_pages < 0) return cs::api_fail(CS_EINVAL, "need_pages < 0");
  for (int32_t i = 0; i < n; ++i)
    if (used_pages[i] < 0 || free_pages[i] < 0) return cs::api_fail(CS_EINVAL, "negative page count");
  const int32_t d = cs::least_occupied(n, used_pages, free_pages, need_pages);
  *decoder = d;
  if (d < 0) return cs::api_fail(CS_ENOMEM, "no decoder has enough free pages");
  return CS_OK;
}

cs_status cs_sched_create(const cs_prefill_curve* curve, double max_wait_s, int32_t n_decoders,
                          cs_pool* const* decoders, cs_sched** out) {
  if (!curve || !out) return cs::api_fail(CS_EINVAL, "null argument");
  if (n_decoders < 0) return cs::api_fail(CS_EINVAL, "n_decoders < 0");
  if (n_decoders > 0 && !decoders) return cs::api_fail(CS_EINVAL, "null decoder array");
  if (!(max_wait_s >= 0) || !std::isfinite(max_wait_s))
    return cs::api_fail(CS_EINVAL, "max_wait_s must be finite and >= 0");
  for (int32_t i = 0; i < n_decoders; ++i)
    if (!decoders[i]) return cs::api_fail(CS_EINVAL, "null decoder pool");
  cs::PrefillCurve c;
  c.c0 = curve->c0;
  c.c1 = curve->c1;
  c.c2 = curve->c2;
  cs_sched* s = new (std::nothrow) cs_sched(c, max_wait_s);
  if (!s) return cs::api_fail(CS_ENOMEM, "out of host memory");
  if (n_decoders > 0) s->decoders.assign(decoders, decoders + n_decoders);
  *out = s;
  return CS_OK;
}

cs_status cs_sched_destroy(cs_sched* sched) {
  if (!sched) return cs::api_fail(CS_EINVAL, "null scheduler");
  delete sched;
  return CS_OK;
}

cs_status cs_sched_admit(cs_sched* sched, int64_t turn1_tokens, double now_s, double* start_s,
                         double* done_s) {
  if (!sched) return cs::api_fail(CS_EINVAL, "null scheduler");
  if (turn1_tokens < 1) return cs::api_fail(CS_EINVAL, "turn1_tokens < 1");
  if (!std::isfinite(now_s)) return cs::api_fail(CS_EINVAL, "now_s not finite");
  if (!sched->admission.admit(turn1_tokens, now_s, start_s, done_s))
    return cs::api_fail(CS_EBUSY, "prefiller saturated: expected wait exceeds max_wait_s");
  return CS_OK;
}

cs_status cs_sched_bind(cs_sched* sched, int64_t kv_tokens, int32_t* decoder) {
  if (!sched || !decoder) return cs::api_fail(CS_EINVAL, "null argument");
  if (kv_tokens < 1) return cs::api_fail(CS_EINVAL, "kv_tokens < 1");
  const int32_t n = static_cast<int32_t>(sched->decoders.size());
  if (n == 0) return cs::api_fail(CS_EINVAL, "the scheduler has no decoder pools (admission only)");
  std::vector<int64_t> used(n), free_(n);
  for (int32_t i = 0; i < n; ++i) {
    const cs_status st = cs_pool_occupancy(sched->decoders[i], &used[i], &free_[i]);
    if (st != CS_OK) return st;
  }
  const int32_t d = cs::least_occupied(n, used.data(), free_.data(), cs::pages_for(kv_tokens));
  *decoder = d;
  if (d < 0) return cs::api_fail(CS_ENOMEM, "no decoder has enough free pages");
  return CS_OK;
}

}  // extern "C"
