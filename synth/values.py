"""Seeded, counter-based synthetic tensor values shared by the tests, the bench and the oracle checks.

This module holds no attention arithmetic: it only turns (key, element index) into a bf16 value, so
any slice of any synthetic tensor can be regenerated bit-for-bit on the host (for the oracle) or on
the device (to fill large inputs quickly).

Generator
---------
* Element index -> 64-bit hash with the SplitMix64 output function (Steele, Lea and Flood,
  "Fast Splittable Pseudorandom Number Generators", OOPSLA 2014): the counter is
  ``key + idx * 0x9E3779B97F4A7C15`` (mod 2^64) and is passed through the published finaliser.
* Approximately N(0, 1): the four 16-bit fields of the hash are summed (Irwin-Hall with n = 4, an
  integer in [0, 262140]); the mean 131070 is subtracted (exact) and the result is multiplied, in
  fp32, by 1/std = sqrt(3)/65536 (std of a sum of four uniform 16-bit integers is ~65536/sqrt(3)).
* Optional per-head scale, multiplied in fp32.
* Rounded once to bf16 with round-to-nearest-even by integer bit arithmetic.

Every step is an integer op or a single IEEE fp32 multiply, so torch on CPU, torch on the GPU and
the numpy reference below produce identical bits (checked in the tests).
"""
from __future__ import annotations

import math

import numpy as np
import torch

_GOLDEN = 0x9E3779B97F4A7C15
_C1 = 0xBF58476D1CE4E5B9
_C2 = 0x94D049BB133111EB
_M64 = (1 << 64) - 1

# fp32 constant 1/std of the Irwin-Hall(4) sum of 16-bit uniforms.
INV_STD_F32 = float(np.float32(math.sqrt(3.0) / 65536.0))
IH_MEAN = 2 * 65535  # mean of the sum of four uniform integers in [0, 65535]


def signed_key(c: int) -> int:
    """A 64-bit stream key as the int64 value with the same bits (for int64 key arrays)."""
    return _s64(c)


def _s64(c: int) -> int:
    """Unsigned 64-bit constant -> the int64 value with the same bits."""
    c &= _M64
    return c - (1 << 64) if c >= (1 << 63) else c


def mix_key(*parts: int) -> int:
    """Derive a 64-bit stream key from integers (seed, conversation, tensor kind, layer, ...)."""
    h = 0x243F6A8885A308D3
    for p in parts:
        h = _splitmix_scalar((h ^ (int(p) & _M64)) & _M64)
    return h


def _splitmix_scalar(x: int) -> int:
    x = (x + _GOLDEN) & _M64
    x ^= x >> 30
    x = (x * _C1) & _M64
    x ^= x >> 27
    x = (x * _C2) & _M64
    x ^= x >> 31
    return x


# ----------------------------------------------------------------------------------------------
# torch implementation (CPU or GPU); int64 arithmetic wraps like uint64 in two's complement.
# ----------------------------------------------------------------------------------------------
def _lsr(x: torch.Tensor, s: int) -> torch.Tensor:
    return (x >> s) & ((1 << (64 - s)) - 1)


def _hash_t(key: int, idx: torch.Tensor) -> torch.Tensor:
    x = idx * _s64(_GOLDEN) + _s64(key)
    x = x ^ _lsr(x, 30)
    x = x * _s64(_C1)
    x = x ^ _lsr(x, 27)
    x = x * _s64(_C2)
    return x ^ _lsr(x, 31)


def _f32_to_bf16_bits_t(x: torch.Tensor) -> torch.Tensor:
    """fp32 -> bf16 bit pattern (int32 holding 0..65535), round to nearest even. Inputs finite."""
    b = x.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    b = b + 0x7FFF + ((b >> 16) & 1)
    return ((b >> 16) & 0xFFFF).to(torch.int32)


def normal_f32(key: int, start: int, count: int, device="cpu") -> torch.Tensor:
    """fp32 values of elements [start, start+count) of stream ``key`` (before scaling/rounding)."""
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    h = _hash_t(key, idx)
    s = (h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) + _lsr(h, 48)
    return (s - IH_MEAN).to(torch.float32) * INV_STD_F32


def bf16_tensor(key: int, shape, head_scale=None, head_axis: int = -2, device="cpu",
                start: int = 0, chunk: int = 1 << 26) -> torch.Tensor:
    """A bf16 tensor of ``shape`` whose flat element e holds stream value ``start + e``.

    ``head_scale`` (1-D fp32, length ``shape[head_axis]``) multiplies each head's values in fp32
    before rounding. Generated in chunks to bound temporaries.
    """
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape)) if shape else 1
    out = torch.empty(n, dtype=torch.int16, device=device)
    if head_scale is not None:
        hs = torch.as_tensor(np.asarray(head_scale, dtype=np.float32), device=device)
        ax = head_axis % len(shape)
        inner = int(np.prod(shape[ax + 1:])) if ax + 1 < len(shape) else 1
        nh = shape[ax]
    for c0 in range(0, n, chunk):
        c1 = min(n, c0 + chunk)
        x = normal_f32(key, start + c0, c1 - c0, device=device)
        if head_scale is not None:
            e = torch.arange(c0, c1, dtype=torch.int64, device=device)
            x = x * hs[(e // inner) % nh]
        out[c0:c1] = _f32_to_bf16_bits_t(x).to(torch.int16)
    return out.view(torch.bfloat16).view(shape)


def bf16_rows(keys, starts, row_len: int, device="cpu") -> torch.Tensor:
    """[R][row_len] bf16: row r holds stream ``keys[r]`` elements ``starts[r] .. +row_len``.

    ``keys``: 64-bit stream keys (Python ints), or an int64 numpy array of their signed bits.

    Same values as ``bf16_tensor`` (unscaled) for the same key and element indices; lets one call
    generate the rows of many conversations / layers at once."""
    if not (isinstance(keys, np.ndarray) and keys.dtype == np.int64):   # int64 arrays: already signed
        keys = np.asarray([_s64(int(k)) for k in keys], dtype=np.int64)
    keys = torch.as_tensor(keys, device=device)
    starts = torch.as_tensor(np.asarray(starts, dtype=np.int64), device=device)
    R = keys.numel()
    if R == 0:
        return torch.empty((0, row_len), dtype=torch.bfloat16, device=device)
    idx = starts[:, None] + torch.arange(row_len, dtype=torch.int64, device=device)[None, :]
    x = idx * _s64(_GOLDEN) + keys[:, None]
    x = x ^ _lsr(x, 30)
    x = x * _s64(_C1)
    x = x ^ _lsr(x, 27)
    x = x * _s64(_C2)
    h = x ^ _lsr(x, 31)
    s = (h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) + _lsr(h, 48)
    f = (s - IH_MEAN).to(torch.float32) * INV_STD_F32
    return _f32_to_bf16_bits_t(f).to(torch.int16).view(torch.bfloat16).view(R, row_len)


# ----------------------------------------------------------------------------------------------
# numpy reference of the same generator (uint64 arithmetic is defined to wrap); used to check the
# torch implementation bit for bit.
# ----------------------------------------------------------------------------------------------
def bf16_bits_numpy(key: int, start: int, count: int, scale: float = 1.0) -> np.ndarray:
    idx = np.arange(start, start + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        x = idx * np.uint64(_GOLDEN) + np.uint64(key)
        x ^= x >> np.uint64(30)
        x *= np.uint64(_C1)
        x ^= x >> np.uint64(27)
        x *= np.uint64(_C2)
        x ^= x >> np.uint64(31)
    m = np.uint64(0xFFFF)
    s = (x & m) + ((x >> np.uint64(16)) & m) + ((x >> np.uint64(32)) & m) + (x >> np.uint64(48))
    f = (s.astype(np.int64) - IH_MEAN).astype(np.float32) * np.float32(INV_STD_F32)
    f = f * np.float32(scale)
    b = f.view(np.uint32).astype(np.uint64)
    b = b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))
    return (b >> np.uint64(16)).astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact upcast of bf16 bit patterns (uint16) to float64."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact upcast of a bf16 torch tensor (any device) to a float64 numpy array."""
    return t.detach().to("cpu").to(torch.float64).numpy()


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns of a bf16 torch tensor as uint16 numpy."""
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)
