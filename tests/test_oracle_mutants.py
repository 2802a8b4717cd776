"""Planted mistakes in a copy of the oracle must be caught by the independent pins (CPU only).

Each mutant is the oracle's source with one plausible slip substituted; the pins that do not depend
on the oracle (brute force, hand-worked example, Q = 0 closed form, GQA repetition) must reject it.
"""
import inspect
import math

import numpy as np
import pytest

import oracle.attention as oa
from tests.test_oracle import brute_attend, _parse_golden_attention

MUTANTS = {
    "diagonal_excluded": ("np.arange(nk)[None, :] <= p[:, None]", "np.arange(nk)[None, :] < p[:, None]"),
    "no_causal_mask": ("np.arange(nk)[None, :] <= p[:, None]", "np.arange(nk)[None, :] >= 0"),
    "scale_1_over_d": ("1.0 / math.sqrt(d)", "1.0 / d"),
    "no_scale": ("1.0 / math.sqrt(d)", "1.0"),
    "gqa_modulo": ("h // (n_q_heads // n_kv_heads)", "h % n_kv_heads"),
    "extend_positions_from_zero": ("np.arange(L - n, L)", "np.arange(0, n)"),
    "unnormalised": ("(w / z) @ v", "w @ v"),
    "keys_as_values": ("(w / z) @ v[:nk, g, :]", "(w / z) @ k[:nk, g, :]"),
}


def _mutant(name):
    src = inspect.getsource(oa)
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, name
    ns = {"__name__": f"mutant_{name}"}
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), ns)
    return ns["attend_last"]


def _pins_pass(attend_last):
    try:
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
    assert _pins_pass(oa.attend_last)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    assert not _pins_pass(_mutant(name)), f"pins failed to catch mutant {name}"
