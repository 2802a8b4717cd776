"""Thin ctypes binding of ``libconserve_attn.so`` (C ABI in include/conserve_attn.h).

Argument marshalling only: shapes, dtypes and devices of torch tensors are checked, their device
pointers and the current HIP stream are passed to the C calls, and negative status codes become
``ConserveError``. Every step of the hot path runs in the library's HIP kernels; there is no
fallback. PyTorch only provides device memory and streams.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libconserve_attn.so")

CS_OK, CS_EINVAL, CS_ENOMEM, CS_ENOENT, CS_ESTATE, CS_ERANGE, CS_EHIP = 0, -1, -2, -3, -4, -5, -6
STATUS_NAMES = {CS_EINVAL: "CS_EINVAL", CS_ENOMEM: "CS_ENOMEM", CS_ENOENT: "CS_ENOENT",
                CS_ESTATE: "CS_ESTATE", CS_ERANGE: "CS_ERANGE", CS_EHIP: "CS_EHIP"}
PAGE_TOKENS = 16

EXPORTS = [
    "cs_pool_kv_bytes", "cs_pool_workspace_bytes", "cs_pool_create", "cs_pool_destroy",
    "cs_pool_occupancy", "cs_conv_create", "cs_conv_destroy", "cs_conv_len", "cs_conv_pages",
    "cs_kv_append", "cs_kv_append_batch", "cs_attn_prefill_turn1", "cs_attn_extend",
    "cs_attn_decode_batch", "cs_mixed_step", "cs_kv_pack_size", "cs_kv_pack", "cs_kv_unpack",
    "cs_profile_start",
    "cs_profile_stop", "cs_last_error",
]
PROFILE_KINDS = ["append", "pack", "unpack", "decode_split", "decode_merge", "attn_fwd"]


class ConserveError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class PoolDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_convs", ctypes.c_int32), ("max_pages_per_conv", ctypes.c_int32),
                ("n_pages", ctypes.c_int64)]


_lib = None


def load_library(path: str = _LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built (there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} not found: build it with `python -m paper_2606_01839_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ, VP = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
    PI32 = ctypes.POINTER(ctypes.c_int32)
    PI64 = ctypes.POINTER(ctypes.c_int64)
    sigs = {
        "cs_pool_kv_bytes": (SZ, [ctypes.POINTER(PoolDesc)]),
        "cs_pool_workspace_bytes": (SZ, [ctypes.POINTER(PoolDesc)]),
        "cs_pool_create": (I32, [ctypes.POINTER(PoolDesc), VP, SZ, VP, SZ, ctypes.c_uint64,
                                 ctypes.POINTER(P)]),
        "cs_pool_destroy": (I32, [P]),
        "cs_pool_occupancy": (I32, [P, PI64, PI64]),
        "cs_conv_create": (I32, [P, PI32]),
        "cs_conv_destroy": (I32, [P, I32]),
        "cs_conv_len": (I32, [P, I32, PI64]),
        "cs_conv_pages": (I32, [P, I32, PI32, I64, PI64]),
        "cs_kv_append": (I32, [P, I32, I32, VP, VP, VP]),
        "cs_kv_append_batch": (I32, [P, I32, PI32, PI32, VP, VP, VP]),
        "cs_attn_prefill_turn1": (I32, [P, I32, PI32, PI32, I32, VP, VP, VP]),
        "cs_attn_extend": (I32, [P, I32, PI32, PI32, I32, VP, VP, VP]),
        "cs_attn_decode_batch": (I32, [P, I32, PI32, I32, VP, VP, VP]),
        "cs_mixed_step": (I32, [P, I32, PI32, PI32, I32, PI32, VP, VP, VP, VP, VP, VP, VP]),
        "cs_kv_pack_size": (I32, [P, I32, ctypes.POINTER(SZ)]),
        "cs_kv_pack": (I32, [P, I32, VP, SZ, VP]),
        "cs_kv_unpack": (I32, [P, VP, SZ, I64, PI32, VP]),
        "cs_profile_start": (I32, [P]),
        "cs_profile_stop": (I32, [P, ctypes.POINTER(ctypes.c_double), PI64]),
        "cs_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    _lib = lib
    return lib


def _check(code: int) -> None:
    if code != CS_OK:
        raise ConserveError(code, _lib.cs_last_error().decode())


def _i32_array(xs):
    a = np.ascontiguousarray(np.asarray(xs, dtype=np.int32).reshape(-1))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _stream_handle(device: torch.device):
    if device.type == "cuda":
        return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)
    return ctypes.c_void_p(0)


def _aligned_bytes(n: int, device: torch.device, align: int = 256) -> torch.Tensor:
    """n bytes of uninitialised memory on `device` starting at an `align`-byte boundary."""
    raw = torch.empty(n + align, dtype=torch.uint8, device=device)
    off = (-raw.data_ptr()) % align
    return raw[off:off + n]


class KVPool:
    """A pool of 16-token KV pages on one GPU, and the conversations that own them.

    Device memory for the pool and its workspace is allocated with torch on ``device``. Method
    names follow the C ABI (cs_<name>).
    """

    def __init__(self, n_layers, n_q_heads, n_kv_heads, head_dim, n_pages, max_convs,
                 max_pages_per_conv, placement_seed=0, device="cuda"):
        self.lib = load_library()
        self.desc = PoolDesc(n_layers, n_q_heads, n_kv_heads, head_dim, max_convs,
                             max_pages_per_conv, n_pages)
        self.device = torch.device(device)
        self.n_layers, self.n_q_heads, self.n_kv_heads, self.head_dim = (
            n_layers, n_q_heads, n_kv_heads, head_dim)
        kvb = self.lib.cs_pool_kv_bytes(ctypes.byref(self.desc))
        wsb = self.lib.cs_pool_workspace_bytes(ctypes.byref(self.desc))
        if kvb == 0 or wsb == 0:
            self._handle = None
            # let cs_pool_create report why the descriptor is invalid
            h = ctypes.c_void_p()
            _check(self.lib.cs_pool_create(ctypes.byref(self.desc), None, 0, None, 0, 0,
                                           ctypes.byref(h)))
        self.kv = _aligned_bytes(kvb, self.device)
        self.ws = _aligned_bytes(wsb, self.device)
        h = ctypes.c_void_p()
        _check(self.lib.cs_pool_create(ctypes.byref(self.desc), self.kv.data_ptr(), kvb,
                                       self.ws.data_ptr(), wsb, placement_seed, ctypes.byref(h)))
        self._handle = h

    # -- lifetime ------------------------------------------------------------------------------
    def close(self):
        if getattr(self, "_handle", None):
            _check(self.lib.cs_pool_destroy(self._handle))
            self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def page_block_bytes(self) -> int:
        return 2 * PAGE_TOKENS * self.head_dim * 2

    def kv_view(self) -> torch.Tensor:
        """The pool as [n_layers][n_pages][n_kv_heads][2*16*head_dim] bf16 bits (int16 view)."""
        return self.kv.view(torch.int16).view(self.n_layers, self.desc.n_pages, self.n_kv_heads,
                                              2 * PAGE_TOKENS * self.head_dim)

    # -- conversations -------------------------------------------------------------------------
    def occupancy(self):
        used, free = ctypes.c_int64(), ctypes.c_int64()
        _check(self.lib.cs_pool_occupancy(self._handle, ctypes.byref(used), ctypes.byref(free)))
        return used.value, free.value

    def conv_create(self) -> int:
        c = ctypes.c_int32()
        _check(self.lib.cs_conv_create(self._handle, ctypes.byref(c)))
        return c.value

    def conv_destroy(self, conv: int) -> None:
        _check(self.lib.cs_conv_destroy(self._handle, conv))

    def conv_len(self, conv: int) -> int:
        n = ctypes.c_int64()
        _check(self.lib.cs_conv_len(self._handle, conv, ctypes.byref(n)))
        return n.value

    def conv_pages(self, conv: int) -> np.ndarray:
        n = ctypes.c_int64()
        code = self.lib.cs_conv_pages(self._handle, conv, None, 0, ctypes.byref(n))
        if code not in (CS_OK, CS_ERANGE):
            _check(code)
        out = np.zeros(n.value, dtype=np.int32)
        _check(self.lib.cs_conv_pages(self._handle, conv,
                                      out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                      n.value, ctypes.byref(n)))
        return out

    # -- tensor checks -------------------------------------------------------------------------
    def _dev(self, t: torch.Tensor, name: str, shape=None) -> int:
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{name} must be bfloat16, got {t.dtype}")
        if t.device != self.device and not (t.device.type == self.device.type == "cuda"
                                            and (t.device.index or 0) == (self.device.index or 0)):
            raise ValueError(f"{name} must be on {self.device}, got {t.device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if shape is not None and tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        return t.data_ptr()

    # -- KV append -----------------------------------------------------------------------------
    def kv_append(self, conv: int, k: torch.Tensor, v: torch.Tensor) -> None:
        """k, v: [n_layers][n_new][n_kv_heads][head_dim] bf16."""
        n = k.shape[1] if k.dim() == 4 else -1
        shp = (self.n_layers, n, self.n_kv_heads, self.head_dim)
        kp, vp = self._dev(k, "k", shp), self._dev(v, "v", shp)
        _check(self.lib.cs_kv_append(self._handle, conv, n, kp, vp, _stream_handle(self.device)))

    def kv_append_batch(self, convs, n_new, k: torch.Tensor, v: torch.Tensor) -> None:
        ca, cp = _i32_array(convs)
        na, npp = _i32_array(n_new)
        if ca.size != na.size:
            raise ValueError("convs and n_new differ in length")
        shp = (self.n_layers, int(na.sum()), self.n_kv_heads, self.head_dim)
        kp, vp = self._dev(k, "k", shp), self._dev(v, "v", shp)
        _check(self.lib.cs_kv_append_batch(self._handle, ca.size, cp, npp, kp, vp,
                                           _stream_handle(self.device)))

    # -- attention -----------------------------------------------------------------------------
    def _attend(self, fn, convs, q_lens, layer, q, out):
        ca, cp = _i32_array(convs)
        qa, qp = _i32_array(q_lens)
        if ca.size != qa.size:
            raise ValueError("convs and q_lens differ in length")
        shp = (int(qa.sum()), self.n_q_heads, self.head_dim)
        qptr = self._dev(q, "q", shp)
        if out is None:
            out = torch.empty(shp, dtype=torch.bfloat16, device=self.device)
        optr = self._dev(out, "out", shp)
        _check(fn(self._handle, ca.size, cp, qp, layer, qptr, optr, _stream_handle(self.device)))
        return out

    def attn_prefill_turn1(self, convs, q_lens, layer, q, out=None) -> torch.Tensor:
        return self._attend(self.lib.cs_attn_prefill_turn1, convs, q_lens, layer, q, out)

    def attn_extend(self, convs, q_lens, layer, q, out=None) -> torch.Tensor:
        return self._attend(self.lib.cs_attn_extend, convs, q_lens, layer, q, out)

    def attn_decode_batch(self, convs, layer, q, out=None) -> torch.Tensor:
        ca, cp = _i32_array(convs)
        shp = (ca.size, self.n_q_heads, self.head_dim)
        qptr = self._dev(q, "q", shp)
        if out is None:
            out = torch.empty(shp, dtype=torch.bfloat16, device=self.device)
        optr = self._dev(out, "out", shp)
        _check(self.lib.cs_attn_decode_batch(self._handle, ca.size, cp, layer, qptr, optr,
                                             _stream_handle(self.device)))
        return out

    def mixed_step(self, ext_convs, ext_lens, dec_convs, k, v, q_ext=None, q_dec=None,
                   out_ext=None, out_dec=None):
        """One decoder step: extend chunks + one decoded token per decoding conversation, appended
        for every layer, then attention of every layer. Returns (out_ext, out_dec)."""
        ea, ep = _i32_array(ext_convs)
        la, lp = _i32_array(ext_lens)
        da, dp = _i32_array(dec_convs)
        if ea.size != la.size:
            raise ValueError("ext_convs and ext_lens differ in length")
        ne, nd, L = int(la.sum()), da.size, self.n_layers
        kv_shape = (L, ne + nd, self.n_kv_heads, self.head_dim)
        kp, vp = self._dev(k, "k", kv_shape), self._dev(v, "v", kv_shape)
        eshape = (L, ne, self.n_q_heads, self.head_dim)
        dshape = (L, nd, self.n_q_heads, self.head_dim)
        qe = qd = oe = od = None
        if ne:
            qe = self._dev(q_ext, "q_ext", eshape)
            if out_ext is None:
                out_ext = torch.empty(eshape, dtype=torch.bfloat16, device=self.device)
            oe = self._dev(out_ext, "out_ext", eshape)
        if nd:
            qd = self._dev(q_dec, "q_dec", dshape)
            if out_dec is None:
                out_dec = torch.empty(dshape, dtype=torch.bfloat16, device=self.device)
            od = self._dev(out_dec, "out_dec", dshape)
        _check(self.lib.cs_mixed_step(self._handle, ea.size, ep, lp, nd, dp, kp, vp, qe, oe, qd, od,
                                      _stream_handle(self.device)))
        return out_ext, out_dec

    # -- instrumentation -----------------------------------------------------------------------
    def profile_start(self) -> None:
        _check(self.lib.cs_profile_start(self._handle))

    def profile_stop(self) -> dict:
        """{kernel kind: (total ms, launches)} for kernels launched since profile_start."""
        n = len(PROFILE_KINDS)
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_int64 * n)()
        _check(self.lib.cs_profile_stop(self._handle, ms, cnt))
        return {k: (ms[i], cnt[i]) for i, k in enumerate(PROFILE_KINDS)}

    # -- one-time transfer ---------------------------------------------------------------------
    def kv_pack_size(self, conv: int) -> int:
        n = ctypes.c_size_t()
        _check(self.lib.cs_kv_pack_size(self._handle, conv, ctypes.byref(n)))
        return n.value

    def kv_pack(self, conv: int, dst: torch.Tensor | None = None) -> torch.Tensor:
        nbytes = self.kv_pack_size(conv)
        if dst is None:
            dst = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        if not dst.is_contiguous() or dst.device.type != self.device.type:
            raise ValueError("dst must be a contiguous tensor on the pool's device")
        _check(self.lib.cs_kv_pack(self._handle, conv, dst.data_ptr(),
                                   dst.numel() * dst.element_size(), _stream_handle(self.device)))
        return dst

    def kv_unpack(self, src: torch.Tensor, n_tokens: int) -> int:
        if not src.is_contiguous() or src.device.type != self.device.type:
            raise ValueError("src must be a contiguous tensor on the pool's device")
        c = ctypes.c_int32()
        _check(self.lib.cs_kv_unpack(self._handle, src.data_ptr(), src.numel() * src.element_size(),
                                     n_tokens, ctypes.byref(c), _stream_handle(self.device)))
        return c.value
