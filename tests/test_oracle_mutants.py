"""Planted mistakes in a copy of the oracle must be caught by the independent pins (CPU only).

Each mutant is the oracle's source with one plausible slip substituted; the pins that do not depend
on the oracle (brute force, hand-worked example, Q = 0 closed form, GQA repetition) must reject it.
"""
import inspect
import math

import numpy as np
import pytest

import oracle.attention as oa
from tests.test_oracle import brute_attend, brute_weights, _parse_golden_attention

MUTANTS = {
    "diagonal_excluded": ("np.arange(nk)[None, :] <= pos[:, None]", "np.arange(nk)[None, :] < pos[:, None]"),
    "no_causal_mask": ("np.arange(nk)[None, :] <= pos[:, None]", "np.arange(nk)[None, :] >= 0"),
    "scale_1_over_d": ("(1.0 / math.sqrt(d))", "(1.0 / d)"),
    "no_scale": ("(1.0 / math.sqrt(d))", "1.0"),
    "scale_doubled": ("(1.0 / math.sqrt(d))", "(2.0 / math.sqrt(d))"),
    "gqa_modulo": ("h // (n_q_heads // n_kv_heads)", "h % n_kv_heads"),
    "extend_positions_from_zero": ("np.arange(L - n, L)", "np.arange(0, n)"),
    "unnormalised": ("return w / z", "return w"),
    "keys_as_values": ("w @ v[: w.shape[1], g, :]", "w @ k[: w.shape[1], g, :]"),
    "max_not_subtracted_per_row": ("m = s.max(axis=1, keepdims=True)", "m = s.max()"),
}


def _mutant(name):
    src = inspect.getsource(oa)
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, name
    ns = {"__name__": f"mutant_{name}"}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)
    return ns


def _weights_pins_pass(weights):
    """Brute-force softmax weights (scale included) and rows summing to 1."""
    rng = np.random.default_rng(3)
    for d, L in [(4, 9), (16, 20)]:
        k = rng.standard_normal((L, d)) * 3
        q = rng.standard_normal((3, d)) * 3
        pos = np.array([L - 1, 0, L // 2])
        w = weights(q, pos, k)
        for i in range(3):
            ref = brute_weights(q[i].tolist(), int(pos[i]), k.tolist())
            if not np.allclose(w[i, : pos[i] + 1], ref, rtol=1e-12, atol=0):
                return False
            if (w[i, pos[i] + 1:] != 0).any() or abs(math.fsum(w[i]) - 1.0) > 1e-12:
                return False
    # rows whose scores lie far apart (one row's exponentials underflow against the other's max)
    k = rng.standard_normal((6, 4)) * 3
    q = np.stack([rng.standard_normal(4), 200 * k[5]])     # second row: score 100 |k5|^2 >> 745
    w = weights(q, np.array([5, 5]), k)
    for i in range(2):
        if not np.allclose(w[i], brute_weights(q[i].tolist(), 5, k.tolist()), rtol=1e-12, atol=0):
            return False
    return True


def _pins_pass(ns):
    attend_last = ns["attend_last"]
    try:
        if not _weights_pins_pass(ns["weights"]):
            return False
        q, k, v, o = _parse_golden_attention()
        if not np.allclose(attend_last(q, k, v), o, atol=1e-12, rtol=0):
            return False
        rng = np.random.default_rng(0)
        for L, n, hq, hkv, d in [(12, 5, 4, 2, 8), (9, 9, 2, 1, 4), (7, 1, 4, 4, 16)]:
            q = rng.standard_normal((n, hq, d))
            k = rng.standard_normal((L, hkv, d))
            v = rng.standard_normal((L, hkv, d))
            ref = brute_attend(q.tolist(), k.tolist(), v.tolist())
            if not np.allclose(attend_last(q, k, v), ref, atol=1e-12, rtol=0):
                return False
            z = attend_last(np.zeros_like(q), k, v)
            for i in range(n):
                for h in range(hq):
                    g = h // (hq // hkv)
                    if not np.allclose(z[i, h], v[: L - n + i + 1, g].mean(0), atol=1e-13):
                        return False
        return True
    except Exception:
        return False


def test_unmutated_oracle_passes_pins():
    assert _pins_pass(vars(oa))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    assert not _pins_pass(_mutant(name)), f"pins failed to catch mutant {name}"
