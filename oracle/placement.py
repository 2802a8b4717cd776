"""Oracle of the conversation-level placement layer: the paper's decoder provisioning rule and
reactive scheduler (arxiv 2606.01839, Section 4), written out plainly in Python.

Test infrastructure only: tests/ and bench.py's CPU baseline may import it; the library never
does. It shares no code with the C++ scheduler (paper_2606_01839_amd/csrc/host/sched.cpp).

- curve_eval: the fitted latency t(L) = c0 + c1 L + c2 L^2.
- prefill_curve_fit: least squares t = c0 + c1 L + c2 L^2 over measured (L, t) samples (Section
  3.1 profiles the prefill latency offline and finds it quadratic in the input length), using
  numpy's least-squares solver on the design matrix [1, x, x^2] of x = L / max|L|.
- provision: Section 4.1. The prefiller saturates at R* = T_p / L_in conversations per second;
  N decoders must satisfy N * T_d >= R * L_d (throughput) and N * B >= R * W (memory) at R = R*;
  N is the smallest integer strictly above both bounds, N = floor(max(bounds)) + 1 (the reading
  adopted for Section 4.1's rule that N exceeds what both inequalities require).
- bind: Section 4.2. A transferred conversation is bound to the decoder with the lowest current
  KV-cache occupancy; readings: occupancy is the fraction of a decoder's pages held by live
  conversations, only decoders with enough free pages for the conversation are candidates, ties go
  to the lower index, and no candidate means the decoder tier is saturated (route elsewhere).
- Admission: Section 4.2. Every turn-1 prefill runs on the prefiller, whose expected work is read
  off the curve; reading: the prefiller is busy until the expected end of the admitted work, a
  new conversation starts at max(arrival, busy_until), and it is refused (routed elsewhere, no
  state change) when its expected wait exceeds a bound.
"""
from __future__ import annotations

import math

import numpy as np

PAGE_TOKENS = 16


def curve_eval(coef, tokens: int) -> float:
    """t(L) = c0 + c1 L + c2 L^2, evaluated as c0 + L (c1 + L c2) in float64."""
    c0, c1, c2 = coef
    L = float(tokens)
    return c0 + L * (c1 + L * c2)


def prefill_curve_fit(tokens, seconds):
    """Least-squares (c0, c1, c2) and the coefficient of determination R^2."""
    L = np.asarray(tokens, dtype=np.float64)
    t = np.asarray(seconds, dtype=np.float64)
    # the columns 1, x, x^2 of x = L / max|L| are well scaled; the solution maps back exactly
    # (c1 = a1 / s, c2 = a2 / s^2) since rescaling columns does not change the least-squares fit
    s = float(np.abs(L).max())
    x = L / s
    A = np.stack([np.ones_like(x), x, x * x], axis=1)
    a, *_ = np.linalg.lstsq(A, t, rcond=None)
    coef = np.array([a[0], a[1] / s, a[2] / (s * s)])
    fitted = A @ a
    ss_res = float(((t - fitted) ** 2).sum())
    ss_tot = float(((t - t.mean()) ** 2).sum())
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else (1.0 if ss_res == 0 else 0.0)
    return tuple(float(x) for x in coef), r2


def provision(prefill_tokens_per_s, mean_turn1_tokens, decoder_tokens_per_s, mean_decoder_tokens,
              convs_per_decoder, mean_lifetime_s):
    """Section 4.1: (R*, throughput bound, memory bound, N)."""
    r_star = prefill_tokens_per_s / mean_turn1_tokens
    n_thr = r_star * mean_decoder_tokens / decoder_tokens_per_s
    n_mem = r_star * mean_lifetime_s / convs_per_decoder
    n = math.floor(max(n_thr, n_mem)) + 1
    return r_star, n_thr, n_mem, n


def pages_for(tokens: int) -> int:
    return -(-tokens // PAGE_TOKENS)


def bind(used_pages, free_pages, need_pages: int) -> int:
    """Index of the least occupied decoder that can hold need_pages more pages, or -1."""
    best = -1
    for i, (u, f) in enumerate(zip(used_pages, free_pages)):
        if f < need_pages:
            continue
        if best < 0:
            best = i
            continue
        cap_i = u + f
        cap_b = used_pages[best] + free_pages[best]
        # exact comparison of the fractions u / cap_i and used_best / cap_b (Python ints)
        if u * cap_b < used_pages[best] * cap_i:
            best = i
    return best


class Admission:
    """The prefiller's expected schedule of admitted turn-1 prefills."""

    def __init__(self, coef, max_wait_s: float):
        self.coef = coef
        self.max_wait = max_wait_s
        self.busy_until = 0.0

    def admit(self, turn1_tokens: int, now_s: float):
        """(start, done) of the admitted prefill, or None when refused (nothing changes)."""
        wait = max(0.0, self.busy_until - now_s)
        if wait > self.max_wait:
            return None
        start = max(now_s, self.busy_until)
        done = start + curve_eval(self.coef, turn1_tokens)
        self.busy_until = done
        return start, done
