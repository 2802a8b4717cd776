// Conversation-level placement over KV page pools: the paper's reactive scheduler (Section 4.2) and
// decoder provisioning rule (Section 4.1). Host-only (no HIP): everything here compiles and is
// tested on a CPU; the C ABI in sched_capi.cpp feeds it the pools' occupancy.
#pragma once

#include <cstdint>

namespace cs {

// Prefill latency as a function of the turn-1 input length (Section 3.1 profiles it offline and
// finds it quadratic): t(L) = c0 + c1 L + c2 L^2 seconds.
struct PrefillCurve {
  double c0 = 0, c1 = 0, c2 = 0;
  double eval(int64_t tokens) const {
    const double L = static_cast<double>(tokens);
    return c0 + L * (c1 + L * c2);
  }
};

// Least-squares fit of t = c0 + c1 L + c2 L^2 to n >= 3 samples with at least three distinct
// lengths. L is scaled by the largest |L| before the fit (conditioning) and the 3x3 normal
// equations are solved by Gaussian elimination with partial pivoting in long double.
// r2 = 1 - SS_res / SS_tot (1 when every sample lies on the curve; SS_tot = 0 gives 1 if the fit is
// exact, else 0). Returns false (out untouched) for too few / degenerate samples.
bool fit_prefill_curve(const int64_t* tokens, const double* seconds, int n, PrefillCurve* out,
                       double* r2);

// Section 4.1: the prefiller saturates at R* = T_p / L_in conversations per second; N decoders
// must satisfy N T_d >= R* L_d (throughput) and N B >= R* W (memory: B conversations fit on one
// decoder, each lives W seconds). n_throughput = R* L_d / T_d, n_memory = R* W / B, and the
// provisioned N is the smallest integer strictly greater than both (the reading adopted for the
// section's rule that N exceeds what both inequalities require). Returns false for non-positive or
// non-finite inputs.
struct Provisioning {
  double saturation_rate = 0;  // R*
  double n_throughput = 0;
  double n_memory = 0;
  int32_t n_decoders = 0;
};
bool provision_decoders(double prefill_tokens_per_s, double mean_turn1_tokens,
                        double decoder_tokens_per_s, double mean_decoder_tokens,
                        double convs_per_decoder, double mean_lifetime_s, Provisioning* out);

// Binding (Section 4.2): among decoders whose free pages cover `need_pages`, the one with the
// lowest occupancy used / (used + free); exact comparison by cross-multiplication, ties to the
// lower index. -1 if no decoder can hold the conversation (decoder pool saturated).
int32_t least_occupied(int32_t n, const int64_t* used_pages, const int64_t* free_pages,
                       int64_t need_pages);

// Admission (Section 4.2): every turn-1 prefill goes to the prefiller; its expected duration is
// read off the curve. The prefiller is modelled as busy until `busy_until` (seconds on the
// caller's clock); a conversation arriving at `now` starts at max(now, busy_until) and ends
// curve(L) later. It is refused (route it elsewhere) when its expected wait max(0, busy_until -
// now) would exceed `max_wait_s`; a refused conversation changes nothing.
class Admission {
 public:
  Admission(PrefillCurve curve, double max_wait_s) : curve_(curve), max_wait_(max_wait_s) {}
  bool admit(int64_t turn1_tokens, double now_s, double* start_s, double* done_s);
  double busy_until() const { return busy_until_; }
  const PrefillCurve& curve() const { return curve_; }

 private:
  PrefillCurve curve_;
  double max_wait_;
  double busy_until_ = 0;
};

}  // namespace cs
