"""Shared helpers for the parity tests: seeded inputs and tolerance checks (the bound of a
bf16-weight kernel's rounding takes the oracle's softmax weights; no kernel arithmetic here)."""
from __future__ import annotations

import math

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


# ---- elementwise bound from the arithmetic of a bf16-weight kernel ------------------------------
# The kernels round every softmax weight to bf16 for the P.V product and sum the same rounded
# weights into the denominator, so their output is an exact convex combination of V with each
# weight perturbed by a relative error of at most delta; then (sum_j w_j (1 + e_j) V_j) /
# (sum_j w_j (1 + e_j)) - O = sum_j w_j e_j (V_j - O) / (1 + sum_j w_j e_j), whose size is at most
# delta / (1 - delta) * sum_j w_j |V_j - O|. delta = 2^-8 (bf16 keeps 8 significant bits, so
# rounding to nearest errs by at most 2^-8 relative) plus the error of
# the fp32 exponent: the score is an fp32 sum of d/16 matrix-core steps and the scale is an fp32
# constant, which perturbs a weight by about ln 2 * (d/16 + 3) * 2^-24 * |score in log2 units|,
# and v_exp_f32 adds ~2^-22 relative. fp32 accumulation of the numerator and denominator over at
# most 4096 keys stays below 2^-12 of the weighted mean |V|, and the output is rounded to bf16
# (half an ulp). Nothing in the bound depends on |O| being small, unlike the fixed max-abs 1e-2.
DELTA_BF16 = 2.0 ** -8
GAMMA_ACC = 2.0 ** -12


def half_ulp_bf16(x: np.ndarray) -> np.ndarray:
    """Half a bf16 ulp at |x| (8 significant bits: ulp = 2^(e - 7) for 2^e <= |x| < 2^(e+1))."""
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -126)))
    return 2.0 ** (e - 8)


def arith_bound(q: np.ndarray, pos, k: np.ndarray, v: np.ndarray, ref: np.ndarray, block: int = 16):
    """Per-element bound (above, without the output rounding) on |kernel - O| for query rows q
    [r][Hq][d] at positions pos against K, V [L][Hkv][d] (float64), ref = the oracle's O."""
    from oracle.attention import kv_head_of, weights
    pos = np.asarray(pos, dtype=np.int64).reshape(-1)
    r, hq, d = q.shape
    hkv = k.shape[1]
    bound = np.zeros_like(ref)
    log2e = 1.0 / math.log(2.0)
    for h in range(hq):
        g = kv_head_of(h, hq, hkv)
        for b0 in range(0, r, block):
            rows = slice(b0, min(r, b0 + block))
            w = weights(q[rows, h], pos[rows], k[:, g])            # [rb][nk], exact zeros masked
            nk = w.shape[1]
            s = np.abs(q[rows, h] @ k[:nk, g].T) * (log2e / math.sqrt(d))
            x = np.where(w > 0, s, 0.0).max(axis=1)
            delta = DELTA_BF16 + math.log(2.0) * (d / 16 + 3) * 2.0 ** -24 * x + 2.0 ** -21
            dev = np.abs(v[None, :nk, g, :] - ref[rows, h][:, None, :])
            mad = np.einsum("rj,rjd->rd", w, dev)
            mabs = w @ np.abs(v[:nk, g])
            bound[rows, h] = (delta / (1 - delta))[:, None] * mad + GAMMA_ACC * mabs
    return bound


def assert_within_arith_bound(got: torch.Tensor, q, pos, k, v, ref: np.ndarray, what: str = ""):
    """Every element of `got` within arith_bound + half a bf16 ulp of the oracle's O."""
    g = f64(got)
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    tol = arith_bound(q, pos, k, v, ref) + half_ulp_bf16(np.maximum(np.abs(ref), np.abs(g)))
    err = np.abs(g - ref)
    worst = np.unravel_index(np.argmax(err / tol), err.shape)
    assert (err <= tol).all(), (f"{what}: |err| {err[worst]:.3e} > bound {tol[worst]:.3e} at {worst} "
                                f"(ref {ref[worst]:.4e}, got {g[worst]:.4e})")
    return float((err / tol).max())


def tile_jumps(q, pos, k, tile=64):
    """Per (row, head): the largest rise, in log2 units, of a key tile's maximum score over the
    maximum of all earlier tiles the row sees."""
    from oracle.attention import kv_head_of
    pos = np.asarray(pos, dtype=np.int64).reshape(-1)
    r, hq, d = q.shape
    hkv = k.shape[1]
    out = np.full((r, hq), -np.inf)
    for h in range(hq):
        s = (q[:, h] @ k[:, kv_head_of(h, hq, hkv)].T) * (1.0 / (math.log(2.0) * math.sqrt(d)))
        for i in range(r):
            row = s[i, : pos[i] + 1]
            n_t = (len(row) + tile - 1) // tile
            mx = [row[t * tile:(t + 1) * tile].max() for t in range(n_t)]
            run = mx[0]
            for t in range(1, n_t):
                out[i, h] = max(out[i, h], mx[t] - run)
                run = max(run, mx[t])
    return out
