// Conversation-level placement: prefill latency curve, decoder provisioning, admission, binding.
#include "host/sched.hpp"

#include <algorithm>
#include <cmath>

namespace cs {

bool fit_prefill_curve(const int64_t* tokens, const double* seconds, int n, PrefillCurve* out,
                       double* r2) {
  if (!tokens || !seconds || !out || n < 3) return false;
  // at least three distinct lengths, all samples finite
  int64_t a = tokens[0], b = tokens[0];
  bool third = false;
  double scale = 0;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(seconds[i])) return false;
    scale = std::max(scale, std::fabs(static_cast<double>(tokens[i])));
    if (tokens[i] != a && b == a) b = tokens[i];
    else if (tokens[i] != a && tokens[i] != b) third = true;
  }
  if (!third || scale == 0) return false;

  // normal equations in x = L / scale: sum x^(i+j) c_j = sum x^i t
  long double m[3][4] = {};
  for (int k = 0; k < n; ++k) {
    const long double x = static_cast<long double>(tokens[k]) / scale;
    const long double p[3] = {1.0L, x, x * x};
    for (int i = 0; i < 3; ++i) {
      for (int j = 0; j < 3; ++j) m[i][j] += p[i] * p[j];
      m[i][3] += p[i] * static_cast<long double>(seconds[k]);
    }
  }
  for (int col = 0; col < 3; ++col) {
    int piv = col;
    for (int r = col + 1; r < 3; ++r)
      if (std::fabs(static_cast<double>(m[r][col])) > std::fabs(static_cast<double>(m[piv][col]))) piv = r;
    if (m[piv][col] == 0) return false;
    if (piv != col)
      for (int j = 0; j < 4; ++j) std::swap(m[piv][j], m[col][j]);
    for (int r = 0; r < 3; ++r) {
      if (r == col) continue;
      const long double f = m[r][col] / m[col][col];
      for (int j = col; j < 4; ++j) m[r][j] -= f * m[col][j];
    }
  }
  PrefillCurve c;
  c.c0 = static_cast<double>(m[0][3] / m[0][0]);
  c.c1 = static_cast<double>(m[1][3] / m[1][1] / scale);
  c.c2 = static_cast<double>(m[2][3] / m[2][2] / scale / scale);
  if (!std::isfinite(c.c0) || !std::isfinite(c.c1) || !std::isfinite(c.c2)) return false;

  if (r2) {
    long double mean = 0;
    for (int k = 0; k < n; ++k) mean += seconds[k];
    mean /= n;
    long double ss_res = 0, ss_tot = 0;
    for (int k = 0; k < n; ++k) {
      const long double e = seconds[k] - static_cast<long double>(c.eval(tokens[k]));
      const long double d = seconds[k] - mean;
      ss_res += e * e;
      ss_tot += d * d;
    }
    *r2 = ss_tot > 0 ? static_cast<double>(1.0L - ss_res / ss_tot) : (ss_res == 0 ? 1.0 : 0.0);
  }
  *out = c;
  return true;
}

bool provision_decoders(double prefill_tokens_per_s, double mean_turn1_tokens,
                        double decoder_tokens_per_s, double mean_decoder_tokens,
                        double convs_per_decoder, double mean_lifetime_s, Provisioning* out) {
  const double v[6] = {prefill_tokens_per_s, mean_turn1_tokens, decoder_tokens_per_s,
                       mean_decoder_tokens, convs_per_decoder, mean_lifetime_s};
  for (double x : v)
    if (!(x > 0) || !std::isfinite(x)) return false;
  if (!out) return false;
  Provisioning p;
  p.saturation_rate = prefill_tokens_per_s / mean_turn1_tokens;
  p.n_throughput = p.saturation_rate * mean_decoder_tokens / decoder_tokens_per_s;
  p.n_memory = p.saturation_rate * mean_lifetime_s / convs_per_decoder;
  const double need = std::max(p.n_throughput, p.n_memory);
  if (!(need < 2147483646.0)) return false;
  p.n_decoders = static_cast<int32_t>(std::floor(need)) + 1;
  *out = p;
  return true;
}

int32_t least_occupied(int32_t n, const int64_t* used_pages, const int64_t* free_pages,
                       int64_t need_pages) {
  int32_t best = -1;
  for (int32_t i = 0; i < n; ++i) {
    if (free_pages[i] < need_pages) continue;
    if (best < 0) {
      best = i;
      continue;
    }
    // used_i / cap_i < used_best / cap_best  <=>  used_i * cap_best < used_best * cap_i
    const __int128 cap_i = static_cast<__int128>(used_pages[i]) + free_pages[i];
    const __int128 cap_b = static_cast<__int128>(used_pages[best]) + free_pages[best];
    if (static_cast<__int128>(used_pages[i]) * cap_b < static_cast<__int128>(used_pages[best]) * cap_i)
      best = i;
  }
  return best;
}

bool Admission::admit(int64_t turn1_tokens, double now_s, double* start_s, double* done_s) {
  const double wait = std::max(0.0, busy_until_ - now_s);
  if (wait > max_wait_) return false;
  const double start = std::max(now_s, busy_until_);
  const double done = start + curve_.eval(turn1_tokens);
  busy_until_ = done;
  if (start_s) *start_s = start;
  if (done_s) *done_s = done;
  return true;
}

}  // namespace cs
