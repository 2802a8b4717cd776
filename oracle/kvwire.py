"""Oracle: a conversation's KV cache as plain concatenation, and the one-time transfer's wire format.

What it follows
---------------
* Section 1 and Section 2.1: a conversation's KV cache only grows; decode appends one entry per
  generated token, and a later turn appends the entries of its new tokens (Section 3.1).
* Section 4 (design) and Section 5.1: the turn-1 cache is produced on the prefiller and transferred
  exactly once to the decoder the conversation is bound to.

The paper does not fix a wire format (its transfer goes through a KV-cache manager whose layout it
does not state). The format adopted here is header-free, logical page order, 16 tokens per page:

    wire = [layer][logical page][kv head] blocks, each block = K part followed by V^T[d][16]

in bf16 (stored as uint16 bit patterns), token slots >= L of the last page zero. The K part is
d/w sub-blocks of w = min(d, 32) dims, sub-block s = K[16 tokens][dims w*s .. w*s + w - 1]
token-major (for d <= 32 that is simply K[16][d]); V is stored dimension-major (transposed). Size
in bytes: n_layers * ceil(L/16) * Hkv * 2 * 16 * d * 2.

Everything here is byte movement: results are compared bit for bit.
"""
from __future__ import annotations

import numpy as np

PAGE = 16


class ConversationKV:
    """KV of one conversation as contiguous arrays [n_layers][L][Hkv][d] of bf16 bit patterns."""

    def __init__(self, n_layers: int, n_kv_heads: int, head_dim: int):
        self.k = np.zeros((n_layers, 0, n_kv_heads, head_dim), dtype=np.uint16)
        self.v = np.zeros((n_layers, 0, n_kv_heads, head_dim), dtype=np.uint16)

    @property
    def length(self) -> int:
        return self.k.shape[1]

    def append(self, k_new: np.ndarray, v_new: np.ndarray) -> None:
        """Append n new tokens: k_new, v_new are [n_layers][n][Hkv][d] uint16."""
        assert k_new.shape == v_new.shape and k_new.shape[0] == self.k.shape[0]
        self.k = np.concatenate([self.k, k_new.astype(np.uint16)], axis=1)
        self.v = np.concatenate([self.v, v_new.astype(np.uint16)], axis=1)


def wire_bytes(n_layers: int, length: int, n_kv_heads: int, head_dim: int) -> int:
    pages = (length + PAGE - 1) // PAGE
    return n_layers * pages * n_kv_heads * 2 * PAGE * head_dim * 2


def k_sub_width(d: int) -> int:
    """Width w of the K sub-blocks of a block (d must be a multiple of it)."""
    w = min(d, 32)
    assert d % w == 0, "head_dim must be <= 32 or a multiple of 32"
    return w


def serialize(k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """k, v: [n_layers][L][Hkv][d] uint16 -> wire buffer as a flat uint16 array."""
    n_layers, L, hkv, d = k.shape
    w = k_sub_width(d)
    pages = (L + PAGE - 1) // PAGE
    out = np.zeros((n_layers, pages, hkv, 2, PAGE * d), dtype=np.uint16)
    for layer in range(n_layers):
        for p in range(pages):
            t0, t1 = p * PAGE, min(L, (p + 1) * PAGE)
            for h in range(hkv):
                kb = np.zeros((PAGE, d), dtype=np.uint16)
                vb = np.zeros((PAGE, d), dtype=np.uint16)
                kb[: t1 - t0] = k[layer, t0:t1, h]
                vb[: t1 - t0] = v[layer, t0:t1, h]
                # K sub-blocks: [d/w][16 tokens][w dims]
                out[layer, p, h, 0] = kb.reshape(PAGE, d // w, w).transpose(1, 0, 2).reshape(-1)
                out[layer, p, h, 1] = vb.T.reshape(-1)        # dimension-major V columns
    return out.reshape(-1)


def deserialize(wire: np.ndarray, n_layers: int, length: int, n_kv_heads: int, head_dim: int):
    """Inverse of ``serialize``: wire (flat uint16) -> (k, v) [n_layers][L][Hkv][d] uint16."""
    pages = (length + PAGE - 1) // PAGE
    sw = k_sub_width(head_dim)
    w = np.asarray(wire, dtype=np.uint16).reshape(n_layers, pages, n_kv_heads, 2, PAGE * head_dim)
    k = np.zeros((n_layers, length, n_kv_heads, head_dim), dtype=np.uint16)
    v = np.zeros_like(k)
    for layer in range(n_layers):
        for p in range(pages):
            t0, t1 = p * PAGE, min(length, (p + 1) * PAGE)
            for h in range(n_kv_heads):
                kb = w[layer, p, h, 0].reshape(head_dim // sw, PAGE, sw).transpose(1, 0, 2)
                k[layer, t0:t1, h] = kb.reshape(PAGE, head_dim)[: t1 - t0]
                vt = w[layer, p, h, 1].reshape(head_dim, PAGE)
                v[layer, t0:t1, h] = vt.T[: t1 - t0]
    return k, v
