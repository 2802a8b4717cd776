"""Planted mistakes in a copy of the placement oracle must be caught by its independent pins (CPU).

Each mutant is oracle/placement.py with one plausible slip substituted; the pins that do not depend
on the oracle -- the paper's worked provisioning example, hand-derived binding and admission cases,
exact recovery of a known quadratic -- must reject it.
"""
import inspect
import os

import pytest

import oracle.placement as opl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "bind_highest_occupancy": ("if u * cap_b < used_pages[best] * cap_i:", "if u * cap_b > used_pages[best] * cap_i:"),
    "bind_absolute_pages": ("if u * cap_b < used_pages[best] * cap_i:", "if u < used_pages[best]:"),
    "bind_ties_to_last": ("if u * cap_b < used_pages[best] * cap_i:", "if u * cap_b <= used_pages[best] * cap_i:"),
    "bind_ignores_room": ("if f < need_pages:", "if False:"),
    "provision_ceil": ("n = math.floor(max(n_thr, n_mem)) + 1", "n = math.ceil(max(n_thr, n_mem))"),
    "provision_throughput_only": ("n = math.floor(max(n_thr, n_mem)) + 1", "n = math.floor(n_thr) + 1"),
    "provision_ratio_inverted": ("r_star * mean_decoder_tokens / decoder_tokens_per_s",
                                 "r_star * decoder_tokens_per_s / mean_decoder_tokens"),
    "admission_no_queue": ("start = max(now_s, self.busy_until)", "start = now_s"),
    "admission_refuses_at_bound": ("if wait > self.max_wait:", "if wait >= self.max_wait:"),
    "curve_no_quadratic_term": ("A = np.stack([np.ones_like(x), x, x * x], axis=1)",
                                "A = np.stack([np.ones_like(x), x, 0 * x], axis=1)"),
    "curve_wrong_unscaling": ("a[2] / (s * s)", "a[2] / s"),
    "curve_eval_no_constant": ("return c0 + L * (c1 + L * c2)", "return L * (c1 + L * c2)"),
    "curve_eval_no_linear": ("return c0 + L * (c1 + L * c2)", "return c0 + L * (L * c2)"),
    "curve_eval_linear_quadratic": ("return c0 + L * (c1 + L * c2)", "return c0 + L * (c1 + c2)"),
    "curve_eval_swapped_terms": ("return c0 + L * (c1 + L * c2)", "return c0 + L * (c2 + L * c1)"),
}


def _mutant(name):
    src = inspect.getsource(opl)
    old, new = MUTANTS[name]
    assert src.count(old) == 1, name
    ns = {"__name__": f"mutant_{name}"}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)
    return ns


def _golden():
    vals = {}
    for line in open(os.path.join(ROOT, "tests", "golden", "provisioning_worked_example.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            k, v = line.split()
            vals[k] = float(v)
    return vals


def _pins_pass(m):
    try:
        g = _golden()
        r, n_thr, n_mem, n = m["provision"](g["prefill_tokens_per_s"], g["mean_turn1_tokens"],
                                            g["decoder_tokens_per_s"], g["mean_decoder_tokens"], 1e9, 1.0)
        if abs(r - g["saturation_rate"]) > 1e-12 or round(n_thr, 2) != g["n_throughput_printed"] or n != 2:
            return False
        if m["provision"](20000, 10000, 1000, 500, 40, 60) != (2.0, 1.0, 3.0, 4):
            return False
        if m["provision"](5000, 1000, 1000, 500, 1e9, 1)[3] != 3:
            return False
        coef = (0.0123, 4.5e-6, 7.25e-11)
        L = [512, 1024, 4096, 16384, 65536, 131072]
        fit, r2 = m["prefill_curve_fit"](L, [coef[0] + x * coef[1] + x * x * coef[2] for x in L])
        if any(abs(a - b) > 1e-7 * abs(b) for a, b in zip(fit, coef)) or abs(r2 - 1.0) > 1e-12:
            return False
        bind = m["bind"]
        if (bind([30, 10, 20], [70, 90, 80], 5), bind([20, 30], [80, 270], 5), bind([10, 10, 10], [90, 90, 90], 1),
                bind([0, 50], [4, 50], 5), bind([0, 50], [4, 3], 5)) != (1, 1, 0, 1, -1):
            return False
        ev = m["curve_eval"]
        if (ev((1.0, 2.0, 3.0), 10), ev((3.0, -1.0, 0.5), 6), ev((0.5, 0.0, 0.0), 7)) != (321.0, 15.0, 0.5):
            return False
        q = m["Admission"]((0.5, 0.25, 0.125), 2.0)
        if (q.admit(2, 0.0), q.admit(4, 1.0), q.admit(2, 2.0), q.admit(2, 3.0)) != (
                (0.0, 1.5), (1.5, 5.0), None, (5.0, 6.5)):
            return False
        a = m["Admission"]((1.0, 0.0, 0.0), 1.5)
        if (a.admit(100, 0.0), a.admit(100, 0.2), a.admit(100, 0.4)) != ((0.0, 1.0), (1.0, 2.0), None):
            return False
        b = m["Admission"]((1.0, 0.0, 0.0), 1.0)       # a wait equal to the bound is accepted
        if (b.admit(10, 0.0), b.admit(10, 0.0)) != ((0.0, 1.0), (1.0, 2.0)):
            return False
        return True
    except Exception:
        return False


def test_unmutated_placement_oracle_passes_pins():
    assert _pins_pass(vars(opl))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_placement_mutant_is_caught(name):
    assert not _pins_pass(_mutant(name)), f"pins failed to catch mutant {name}"
