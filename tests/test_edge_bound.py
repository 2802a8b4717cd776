"""CPU: the inputs of the hard attention cases and the elementwise tolerance the GPU edge tests use.

* The profiles of ``synth.edge`` really move the running maximum: for ``peak`` and ``rise`` some
  64-key tile raises a row's maximum by more than 8 log2 units over all earlier tiles (the
  condition under which the flash-attention kernels rescale their accumulators after tile 0).
* ``tests.helpers.arith_bound`` holds for a plain CPU model of a bf16-weight kernel (weights rounded
  to bf16, the same rounded weights summed into the denominator, output rounded to bf16) on every
  profile, including outputs far above 4 in magnitude; and it is not vacuous: the same model with
  weights rounded to 5 significant bits instead of 8 breaks it.
"""
import math

import numpy as np
import pytest
import torch

from oracle.attention import attend_rows, kv_head_of
from synth.edge import PROFILES, edge_inputs
from tests.helpers import arith_bound, half_ulp_bf16, tile_jumps

LOG2E = 1.0 / math.log(2.0)


def _f64(t):
    return t.float().numpy().astype(np.float64)


def _inputs(profile, L, n, hq, hkv, d, seed, v_scale=1.0):
    k, v, q = edge_inputs(profile, L, n, hq, hkv, d, lambda h: kv_head_of(h, hq, hkv), seed, v_scale=v_scale)
    return _f64(q), np.arange(L - n, L), _f64(k), _f64(v)


@pytest.mark.parametrize("profile", ["peak", "rise"])
@pytest.mark.parametrize("d", [64, 128])
def test_profiles_move_the_running_max(profile, d):
    q, pos, k, v = _inputs(profile, 700, 700, 4, 2, d, seed=5)
    jumps = tile_jumps(q, pos, k)
    frac = float((jumps > 8).mean())
    assert frac > (0.5 if profile == "rise" else 0.2), frac


def test_zero_profile_is_uniform_weights():
    q, pos, k, v = _inputs("zero", 50, 10, 4, 2, 64, seed=1)
    out = attend_rows(q, pos, k, v)
    for i, p in enumerate(pos):
        for h in range(4):
            np.testing.assert_allclose(out[i, h], v[: p + 1, h // 2].mean(0), atol=1e-14)


def _bf16_round(x, bits=8):
    """Round to `bits` significant bits, nearest even (bits = 8 is bf16)."""
    if bits == 8:
        return torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).double().numpy()
    m, e = np.frexp(x)
    scale = 2.0 ** bits
    return np.ldexp(np.round(m * scale) / scale, e)


def kernel_model(q, pos, k, v, weight_bits=8):
    """CPU model of the kernels' rounding: weights 2^(x - max) rounded, the same rounded weights in
    the numerator and the denominator, the output rounded to bf16."""
    r, hq, d = q.shape
    hkv = k.shape[1]
    out = np.empty((r, hq, d))
    for h in range(hq):
        g = kv_head_of(h, hq, hkv)
        for i in range(r):
            x = (k[: pos[i] + 1, g] @ q[i, h]) * (LOG2E / math.sqrt(d))
            p = _bf16_round(np.exp2(x - x.max()), weight_bits)
            out[i, h] = (p @ v[: pos[i] + 1, g]) / p.sum()
    return _bf16_round(out)


@pytest.mark.parametrize("profile", PROFILES)
@pytest.mark.parametrize("v_scale", [1.0, 64.0])
def test_bound_holds_for_the_rounding_model(profile, v_scale):
    q, pos, k, v = _inputs(profile, 300, 40, 4, 2, 64, seed=7, v_scale=v_scale)
    ref = attend_rows(q, pos, k, v)
    got = kernel_model(q, pos, k, v)
    tol = arith_bound(q, pos, k, v, ref) + half_ulp_bf16(np.maximum(np.abs(ref), np.abs(got)))
    assert (np.abs(got - ref) <= tol).all()
    if v_scale > 1:
        assert np.abs(ref).max() > 4     # the case the fixed max-abs 1e-2 cannot cover


def test_bound_is_not_vacuous():
    """Weights rounded to 5 significant bits (error up to 2^-5) break the bound somewhere."""
    broke = False
    for profile in ("rise", "saw"):
        q, pos, k, v = _inputs(profile, 300, 40, 4, 2, 64, seed=7)
        ref = attend_rows(q, pos, k, v)
        got = kernel_model(q, pos, k, v, weight_bits=5)
        tol = arith_bound(q, pos, k, v, ref) + half_ulp_bf16(np.maximum(np.abs(ref), np.abs(got)))
        broke |= bool((np.abs(got - ref) > tol).any())
    assert broke
