"""Structured inputs for the hard cases of causal softmax attention (seeded, host side).

The unit-variance generator in ``synth.values`` gives scores of a few units, so a flash-attention
kernel's running maximum is set by its first key tile and never has to move much afterwards. The
profiles below make it move, each for a different reason; they hold no attention arithmetic, only
the construction of Q, K and V:

* ``peak``: query row i of head h is ``alpha * K[j*]`` for a key j* drawn uniformly from the keys
  the row sees, with alpha a power of two (exact in bf16), so one key dominates the row's
  softmax by tens of log2 units and it can sit in any key tile.
* ``rise``: every key is ``ramp(j) * u + noise`` along one fixed direction u (entries +-1) and every
  query is ``u + noise``, so scores climb by about ``slope`` log2 units per key: each new key tile
  raises the row maximum far past the old one.
* ``saw``: the same ramp restarted every ``period`` keys: the maximum climbs inside a tooth and
  drops at the next, so later tiles also bring keys far below the running maximum.
* ``zero``: Q = 0, so every visible key has the same weight (the running mean of V).

``v_scale`` multiplies V by a power of two (exact in bf16) to reach outputs of large magnitude.
Everything is drawn in float32 with numpy's PCG64 and rounded once to bf16 (round to nearest
even); the returned tensors are what both the GPU path and the oracle consume.
"""
from __future__ import annotations

import math

import numpy as np
import torch

PROFILES = ("peak", "rise", "saw", "zero")


def _bf16(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)


def edge_inputs(profile: str, L: int, n_q: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                kv_of_head, seed: int, v_scale: float = 1.0, alpha: float = 4.0,
                slope: float = 10.0 / 64.0, period: int = 192):
    """K, V [L][Hkv][d] and Q [n_q][Hq][d] (bf16, CPU) for the last n_q positions of a
    conversation of L tokens. ``kv_of_head(h)`` names the KV head query head h reads (used by
    ``peak`` to aim a query at one of its own keys)."""
    if profile not in PROFILES:
        raise ValueError(f"unknown profile {profile!r}")
    assert 0 < n_q <= L
    rng = np.random.default_rng(seed)
    d = head_dim
    v = rng.standard_normal((L, n_kv_heads, d)).astype(np.float32) * np.float32(v_scale)
    if profile in ("rise", "saw"):
        u = np.where(rng.integers(0, 2, size=d) == 1, 1.0, -1.0).astype(np.float32)
        j = np.arange(L)
        t = j % period if profile == "saw" else j
        # a score along u is ramp * d / sqrt(d) = ramp * sqrt(d) natural units, i.e. ramp * sqrt(d)
        # * log2(e) log2 units: ramp = slope * t * ln 2 / sqrt(d) climbs `slope` log2 units per key
        ramp = (slope * t * math.log(2.0) / math.sqrt(d)).astype(np.float32)
        k = ramp[:, None, None] * u[None, None, :] + \
            np.float32(0.25) * rng.standard_normal((L, n_kv_heads, d)).astype(np.float32)
        q = u[None, None, :] + np.float32(0.1) * rng.standard_normal((n_q, n_q_heads, d)).astype(np.float32)
        return _bf16(k), _bf16(v), _bf16(q)
    k = rng.standard_normal((L, n_kv_heads, d)).astype(np.float32)
    if profile == "zero":
        return _bf16(k), _bf16(v), torch.zeros((n_q, n_q_heads, d), dtype=torch.bfloat16)
    # peak: the bf16 keys are what the query is aimed at, so round K first
    kb = _bf16(k)
    kf = kb.float().numpy()
    q = np.empty((n_q, n_q_heads, d), dtype=np.float32)
    for i in range(n_q):
        pos = L - n_q + i
        for h in range(n_q_heads):
            jstar = int(rng.integers(0, pos + 1))
            q[i, h] = np.float32(alpha) * kf[jstar, kv_of_head(h)]
    return kb, _bf16(v), _bf16(q)
