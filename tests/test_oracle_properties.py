"""Property pins of the CPU oracle's attention (no GPU), on random shapes drawn by hypothesis.

Each property is an identity of softmax(q k^T / sqrt(d)) V that holds exactly in real arithmetic
(fp64 here, compared to 1e-10), and each fails for a plausible slip in the oracle:
* V -> a V + c gives O -> a O + c (the weights of a row sum to 1): an unnormalised or wrongly
  normalised softmax, or a denominator over other keys than the numerator, breaks it;
* k_j -> k_j + u for every key j shifts every score of a row by the same q . u, which a softmax
  ignores: a missing max subtraction still passes, but a per-key slip (a score compared across
  rows, a mask applied after the normalisation) does not;
* q -> t q with k -> k / t leaves every score unchanged: a slip that treats queries and keys
  differently (a norm or an offset applied to one side only) breaks it;
* keys and values after a row's position never change that row (the causal mask);
* the last row, which sees every key, is invariant to permuting the keys together with their
  values.
"""
import inspect

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle.attention as oa
from oracle.attention import attend_last, attend_rows

SHAPES = st.sampled_from([(1, 1, 4), (2, 1, 8), (4, 2, 8), (4, 4, 16), (8, 2, 16)])


def _case(seed, L, n, shape, scale=1.0):
    hq, hkv, d = shape
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((n, hq, d)) * scale
    k = rng.standard_normal((L, hkv, d)) * scale
    v = rng.standard_normal((L, hkv, d))
    return rng, q, k, v


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), L=st.integers(1, 40), shape=SHAPES,
       a=st.floats(-8, 8, allow_nan=False), c=st.floats(-100, 100, allow_nan=False))
def test_values_affine_map_passes_through(seed, L, shape, a, c):
    rng, q, k, v = _case(seed, L, L, shape)
    shift = rng.standard_normal(shape[2]) * c
    got = attend_last(q, k, a * v + shift)
    want = a * attend_last(q, k, v) + shift
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10 * (1 + abs(c)))


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), L=st.integers(1, 40), shape=SHAPES,
       scale=st.floats(0.1, 3.0))
def test_common_key_offset_changes_nothing(seed, L, shape, scale):
    rng, q, k, v = _case(seed, L, L, shape, scale)
    u = rng.standard_normal((k.shape[1], k.shape[2])) * 4.0     # one offset per kv head
    np.testing.assert_allclose(attend_last(q, k + u[None], v), attend_last(q, k, v), rtol=1e-9, atol=1e-10)


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), L=st.integers(1, 40), shape=SHAPES,
       t=st.floats(0.25, 4.0))
def test_query_key_rescaling_changes_nothing(seed, L, shape, t):
    _, q, k, v = _case(seed, L, L, shape)
    np.testing.assert_allclose(attend_last(q * t, k / t, v), attend_last(q, k, v), rtol=1e-9, atol=1e-10)


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), L=st.integers(2, 40), extra=st.integers(1, 20), shape=SHAPES)
def test_keys_after_a_row_do_not_reach_it(seed, L, extra, shape):
    rng, q, k, v = _case(seed, L + extra, L, shape)
    pos = rng.integers(0, L, size=6)
    qr = rng.standard_normal((6, shape[0], shape[2]))
    base = attend_rows(qr, pos, k[:L], v[:L])
    k2, v2 = k.copy(), v.copy()
    k2[L:] = rng.standard_normal(k2[L:].shape) * 50.0
    v2[L:] = rng.standard_normal(v2[L:].shape) * 50.0
    np.testing.assert_array_equal(attend_rows(qr, pos, k2, v2), base)


@settings(max_examples=40, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), L=st.integers(1, 40), shape=SHAPES)
def test_last_row_invariant_to_key_order(seed, L, shape):
    rng, q, k, v = _case(seed, L, 1, shape)
    perm = rng.permutation(L)
    np.testing.assert_allclose(attend_last(q, k[perm], v[perm]), attend_last(q, k, v), rtol=1e-10, atol=1e-12)


# ---- the properties reject planted slips (a mutated copy of the oracle's source) -------------------
def _properties_hold(last, rows):
    """The five properties above on fixed seeds, for attention functions `last` / `rows`."""
    ok = True
    for seed, L, shape in [(1, 9, (4, 2, 8)), (2, 23, (2, 1, 16)), (3, 5, (1, 1, 4))]:
        rng, q, k, v = _case(seed, L, L, shape)
        shift = rng.standard_normal(shape[2]) * 30.0
        ok &= np.allclose(last(q, k, -2.5 * v + shift), -2.5 * last(q, k, v) + shift, rtol=1e-9, atol=1e-8)
        u = rng.standard_normal((shape[1], shape[2])) * 4.0
        ok &= np.allclose(last(q, k + u[None], v), last(q, k, v), rtol=1e-9, atol=1e-10)
        ok &= np.allclose(last(q * 3.0, k / 3.0, v), last(q, k, v), rtol=1e-9, atol=1e-10)
        pos = rng.integers(0, L - 2, size=4) if L > 3 else np.zeros(4, dtype=np.int64)
        k2, v2 = k.copy(), v.copy()
        k2[-2:] *= 50.0
        v2[-2:] *= 50.0
        ok &= np.array_equal(rows(q[:4], pos, k2, v2), rows(q[:4], pos, k, v)) if L >= 4 else True
        perm = rng.permutation(L)
        ok &= np.allclose(last(q[-1:], k[perm], v[perm]), last(q[-1:], k, v), rtol=1e-10, atol=1e-12)
    return bool(ok)


PROPERTY_MUTANTS = {
    "unnormalised": [("return w / z", "return w")],
    "mask_after_normalisation": [("s = np.where(visible, s, -np.inf)", "s = s"),
                                 ("return w / z", "return np.where(visible, w / z, 0.0)")],
    "query_normalised": [("s = (q_rows @ k_head[:nk].T)",
                          "s = ((q_rows / np.linalg.norm(q_rows, axis=1, keepdims=True)) @ k_head[:nk].T)")],
    "position_dependent_weight": [("w = np.exp(s - m)", "w = np.exp(s - m - 0.01 * np.arange(nk)[None, :])")],
}


def _mutant(name):
    src = inspect.getsource(oa)
    for old, new in PROPERTY_MUTANTS[name]:
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
    ns = {"__name__": f"mutant_{name}"}
    exec(compile(src, f"<mutant {name}>", "exec"), ns)
    return ns


def test_properties_hold_for_the_oracle():
    assert _properties_hold(attend_last, attend_rows)


@pytest.mark.parametrize("name", sorted(PROPERTY_MUTANTS))
def test_properties_reject_mutant(name):
    ns = _mutant(name)
    with np.errstate(all="ignore"):
        assert not _properties_hold(ns["attend_last"], ns["attend_rows"]), name
