"""Seeded synthetic agentic conversation traces (lengths only; values come from ``synth.values``).

The paper's workload is agentic traces whose first turn is a long prompt ("tens of thousands" of
tokens) followed by many short appended tool outputs and decodes (Section 3, Fig. 1; mean about 15k
input and 1k output tokens per conversation, Section 5.1). Those traces are not available, so the
five workloads below are synthetic stand-ins with the shapes the hot path is measured on. Lengths
are drawn on the host with numpy's PCG64; every draw is listed here so a trace is reproducible from
its seed alone.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PAGE = 16


@dataclass(frozen=True)
class Shape:
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def kv_bytes_per_token_layer(self) -> int:
        return 2 * self.n_kv_heads * self.head_dim * 2


TINY = Shape(n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64)
LLAMA8B_1L = Shape(n_layers=1, n_q_heads=32, n_kv_heads=8, head_dim=128)
LLAMA8B = Shape(n_layers=32, n_q_heads=32, n_kv_heads=8, head_dim=128)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _lognormal_int(rng, median, sigma, lo, hi, size):
    x = np.exp(rng.normal(np.log(median), sigma, size=size))
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


# ---------------------------------------------------------------------------------------------
# 1. tiny oracle-sized trace
# ---------------------------------------------------------------------------------------------
@dataclass(frozen=True)
class TinyTrace:
    """2 conversations x 3 turns; turn 1 = 256-token prefill, then (after the one-time transfer)
    16 single-token decodes; turns 2-3 append 32 tokens then decode 16. 4q/2kv heads, d = 64."""
    seed: int = 1001
    shape: Shape = TINY
    n_convs: int = 2
    turn1: int = 256
    append: int = 32
    decodes: int = 16
    turns: int = 3
    turn1_decode: bool = True

    def final_len(self) -> int:
        n = self.turn1 + (self.decodes if self.turn1_decode else 0)
        return n + (self.turns - 1) * (self.append + self.decodes)


# ---------------------------------------------------------------------------------------------
# 2. decode-only batch
# ---------------------------------------------------------------------------------------------
@dataclass(frozen=True)
class DecodeBatch:
    seed: int = 1002
    shape: Shape = LLAMA8B_1L
    batch: int = 64
    lo: int = 8192
    hi: int = 32768
    scale_lo: float = 0.5
    scale_hi: float = 2.0

    def lengths(self) -> np.ndarray:
        return _rng(self.seed).integers(self.lo, self.hi, size=self.batch, endpoint=True)

    def head_scales(self):
        """(s_K, s_V): independent fp32 scales per KV head, uniform in [scale_lo, scale_hi]."""
        r = _rng(self.seed + 7919)
        h = self.shape.n_kv_heads
        sk = r.uniform(self.scale_lo, self.scale_hi, size=h).astype(np.float32)
        sv = r.uniform(self.scale_lo, self.scale_hi, size=h).astype(np.float32)
        return sk, sv


# ---------------------------------------------------------------------------------------------
# 3. incremental extend-prefill
# ---------------------------------------------------------------------------------------------
@dataclass(frozen=True)
class ExtendBatch:
    seed: int = 1003
    shape: Shape = LLAMA8B_1L
    n_convs: int = 16
    prefix_lo: int = 16384
    prefix_hi: int = 65536
    chunk_median: int = 1024
    chunk_sigma: float = 0.7
    chunk_lo: int = 128
    chunk_hi: int = 4096

    def lengths(self):
        r = _rng(self.seed)
        prefix = r.integers(self.prefix_lo, self.prefix_hi, size=self.n_convs, endpoint=True)
        chunk = _lognormal_int(r, self.chunk_median, self.chunk_sigma, self.chunk_lo,
                               self.chunk_hi, self.n_convs)
        return prefix, chunk


# ---------------------------------------------------------------------------------------------
# 4. turn-1 prefill + one-time transfer
# ---------------------------------------------------------------------------------------------
@dataclass(frozen=True)
class PrefillTransfer:
    seed: int = 1004
    shape: Shape = LLAMA8B_1L
    n_convs: int = 8
    lo: int = 32768
    hi: int = 131072
    dst_seed: int = 2004

    def lengths(self) -> np.ndarray:
        return _rng(self.seed).integers(self.lo, self.hi, size=self.n_convs, endpoint=True)


# ---------------------------------------------------------------------------------------------
# 5. mixed agentic trace
# ---------------------------------------------------------------------------------------------
@dataclass
class Conversation:
    cid: int
    turn1: int
    appends: list = field(default_factory=list)  # turn 2.. append lengths
    decodes: list = field(default_factory=list)  # decodes per turn (len = turns)

    @property
    def turns(self) -> int:
        return len(self.decodes)

    def final_len(self) -> int:
        return self.turn1 + sum(self.appends) + sum(self.decodes)


@dataclass(frozen=True)
class MixedTrace:
    seed: int = 1005
    shape: Shape = LLAMA8B
    n_convs: int = 256
    turns_lo: int = 5
    turns_hi: int = 30
    turn1_median: int = 8192
    turn1_sigma: float = 1.0
    turn1_lo: int = 1024
    turn1_hi: int = 65536
    append_median: int = 1024
    append_sigma: float = 0.7
    append_lo: int = 16
    append_hi: int = 16384
    decode_median: int = 200
    decode_sigma: float = 0.7
    decode_lo: int = 1
    decode_hi: int = 4096

    def conversations(self) -> list:
        r = _rng(self.seed)
        turns = r.integers(self.turns_lo, self.turns_hi, size=self.n_convs, endpoint=True)
        t1 = _lognormal_int(r, self.turn1_median, self.turn1_sigma, self.turn1_lo, self.turn1_hi,
                            self.n_convs)
        out = []
        for c in range(self.n_convs):
            k = int(turns[c])
            app = _lognormal_int(r, self.append_median, self.append_sigma, self.append_lo,
                                 self.append_hi, k - 1)
            dec = _lognormal_int(r, self.decode_median, self.decode_sigma, self.decode_lo,
                                 self.decode_hi, k)
            out.append(Conversation(c, int(t1[c]), [int(a) for a in app], [int(d) for d in dec]))
        return out


def pages_for(n_tokens: int) -> int:
    return (int(n_tokens) + PAGE - 1) // PAGE


# Stream keys for synthetic tensors: a tensor of conversation c, kind k, layer l in workload w is
# generated from key mix_key(seed, c, k, l); element (pos, head, dim) has index (pos*H + head)*d + dim,
# so a conversation's values at a position never depend on how its tokens were batched.
KIND_Q, KIND_K, KIND_V = 1, 2, 3
