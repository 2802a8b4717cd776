"""Oracle: causal scaled-dot-product attention over a conversation's contiguous KV (float64).

What it follows
---------------
* Section 2.1 (LLM Serving Techniques): prefill produces a KV entry for every prompt token; a decode
  step reads the full KV cache and appends one new entry.
* Section 3.1 (prefix caching paragraph) and Section 4 (design): a later turn computes KV only for
  its appended tokens and attends against the whole cached history of the conversation.
* The attention itself is the scaled dot-product attention of the Transformer the paper serves
  (its reference "transformer", Vaswani et al. 2017): softmax(q k^T / sqrt(d)) V.

Readings where the paper is silent (each one is listed in the design doc):
* Append-then-attend: a query at absolute position p sees keys 0..p, itself included, for turn-1
  prefill, extend and decode alike.
* Scale exactly 1/sqrt(d); no soft-cap, ALiBi, window or rotary embedding.
* Grouped-query heads: query head h reads KV head h // (Hq / Hkv).

All arithmetic is float64. Inputs are float64 arrays (exact upcasts of the bf16 values the GPU sees).
"""
from __future__ import annotations

import math

import numpy as np


def kv_head_of(h: int, n_q_heads: int, n_kv_heads: int) -> int:
    """GQA map: contiguous groups of Hq/Hkv query heads share one KV head."""
    return h // (n_q_heads // n_kv_heads)


def weights(q_rows: np.ndarray, pos, k_head: np.ndarray) -> np.ndarray:
    """Softmax weights of query rows of one head over the keys of its KV head (steps 1-2 below).

    q_rows: [r][d] float64 query rows; pos: [r] absolute positions; k_head: [>= max(pos)+1][d]
    float64 keys of the row's KV head. Returns [r][max(pos)+1] float64: row i holds
    softmax_j(q_i . k_j / sqrt(d)) over the visible keys j <= pos[i] and exact zeros for the keys
    past pos[i] (the causal mask). The maximum is subtracted before exponentiating (a stable
    softmax; the result is mathematically the same).
    """
    q_rows = np.asarray(q_rows, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.int64).reshape(-1)
    d = q_rows.shape[-1]
    nk = int(pos.max()) + 1
    s = (q_rows @ k_head[:nk].T) * (1.0 / math.sqrt(d))               # step 1: scores
    visible = np.arange(nk)[None, :] <= pos[:, None]
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)                                    # step 2: stable softmax
    w = np.exp(s - m)
    z = w.sum(axis=1, keepdims=True)
    return w / z


def attend_rows(q: np.ndarray, pos, k: np.ndarray, v: np.ndarray, block: int = 256) -> np.ndarray:
    """Attention output for query rows at the given absolute positions.

    q:   [r][Hq][d] float64 query rows.
    pos: [r] absolute positions (row i sees keys 0..pos[i]).
    k,v: [L][Hkv][d] float64, the conversation's contiguous keys/values (L > max(pos)).
    Returns [r][Hq][d] float64.

    Rows are evaluated in groups of ``block`` only to bound the size of the score matrix; every row
    is the same formula on its own keys.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.int64).reshape(-1)
    r, hq, d = q.shape
    hkv = k.shape[1]
    if r == 0:
        return np.zeros((0, hq, d))
    assert hq % hkv == 0 and k.shape[2] == d and v.shape == k.shape
    assert pos.shape[0] == r and pos.min() >= 0 and pos.max() < k.shape[0]
    out = np.empty((r, hq, d), dtype=np.float64)
    for h in range(hq):
        g = kv_head_of(h, hq, hkv)
        for b0 in range(0, r, block):
            rows = slice(b0, min(r, b0 + block))
            w = weights(q[rows, h, :], pos[rows], k[:, g, :])
            out[rows, h, :] = w @ v[: w.shape[1], g, :]                  # step 3: weighted values
    return out


def attend_last(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Attention for the last n = q.shape[0] positions of a conversation of length L = k.shape[0].

    Turn-1 prefill is n == L, extend is n < L, decode is n == 1.
    """
    n, L = q.shape[0], k.shape[0]
    assert 0 <= n <= L
    return attend_rows(q, np.arange(L - n, L), k, v)
