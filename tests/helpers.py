"""Shared helpers for the parity tests: seeded inputs and tolerance checks (no method arithmetic)."""
from __future__ import annotations

import numpy as np
import torch

from synth import values as sv
from synth.traces import KIND_K, KIND_Q, KIND_V

ATOL_MAX = 1e-2   # max-abs error allowed on an attention output tensor
RTOL_L2 = 3e-3    # relative L2 error allowed on an attention output tensor


def kv_tokens(seed, conv, layer_count, start, n, n_kv_heads, head_dim, k_scale=None, v_scale=None,
              device="cpu"):
    """K and V of tokens [start, start+n) of a conversation: [n_layers][n][Hkv][d] bf16.

    Values are addressed by (position, head, dim), so any slice regenerates identically."""
    ks, vs = [], []
    for layer in range(layer_count):
        per = n_kv_heads * head_dim
        ks.append(sv.bf16_tensor(sv.mix_key(seed, conv, KIND_K, layer), (n, n_kv_heads, head_dim),
                                 head_scale=k_scale, start=start * per, device=device))
        vs.append(sv.bf16_tensor(sv.mix_key(seed, conv, KIND_V, layer), (n, n_kv_heads, head_dim),
                                 head_scale=v_scale, start=start * per, device=device))
    return torch.stack(ks), torch.stack(vs)


def q_tokens(seed, conv, layer, start, n, n_q_heads, head_dim, device="cpu"):
    """Queries of positions [start, start+n) of a conversation: [n][Hq][d] bf16."""
    per = n_q_heads * head_dim
    return sv.bf16_tensor(sv.mix_key(seed, conv, KIND_Q, layer), (n, n_q_heads, head_dim),
                          start=start * per, device=device)


def f64(t: torch.Tensor) -> np.ndarray:
    return sv.bf16_to_f64(t)


def errors(got: torch.Tensor, ref: np.ndarray):
    g = f64(got)
    diff = g - ref
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    den = float(np.sqrt((ref ** 2).sum()))
    rel_l2 = float(np.sqrt((diff ** 2).sum()) / den) if den > 0 else float(np.sqrt((diff ** 2).sum()))
    return max_abs, rel_l2


def assert_close(got: torch.Tensor, ref: np.ndarray, what: str = ""):
    assert tuple(got.shape) == tuple(ref.shape), (what, tuple(got.shape), ref.shape)
    g = f64(got)
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    max_abs, rel_l2 = errors(got, ref)
    assert max_abs <= ATOL_MAX and rel_l2 <= RTOL_L2, f"{what}: max_abs={max_abs:.3e} rel_l2={rel_l2:.3e}"
    return max_abs, rel_l2
