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

CS_OK, CS_EINVAL, CS_ENOMEM, CS_ENOENT, CS_ESTATE, CS_ERANGE, CS_EHIP, CS_EBUSY = 0, -1, -2, -3, -4, -5, -6, -7
CS_MIXED_LAYER_ORDERED = 1   # cs_mixed_step flag: layer l+1 starts after layer l
STATUS_NAMES = {CS_EINVAL: "CS_EINVAL", CS_ENOMEM: "CS_ENOMEM", CS_ENOENT: "CS_ENOENT",
                CS_ESTATE: "CS_ESTATE", CS_ERANGE: "CS_ERANGE", CS_EHIP: "CS_EHIP",
                CS_EBUSY: "CS_EBUSY"}
PAGE_TOKENS = 16
WIRE_FORMAT_VERSION = 1       # CS_WIRE_FORMAT_VERSION: the frozen layout of kv_pack / kv_unpack

EXPORTS = [
    "cs_pool_kv_bytes", "cs_pool_workspace_bytes", "cs_pool_create", "cs_pool_destroy",
    "cs_pool_occupancy", "cs_conv_create", "cs_conv_destroy", "cs_conv_len", "cs_conv_pages",
    "cs_kv_append", "cs_kv_append_batch", "cs_attn_prefill_turn1", "cs_attn_extend",
    "cs_attn_decode_batch", "cs_attn_decode_batch_noalloc", "cs_mixed_step", "cs_kv_pack_size", "cs_kv_pack", "cs_kv_unpack",
    "cs_profile_start",
    "cs_profile_stop", "cs_device_info", "cs_probe_stream_read", "cs_debug_fail_launches",
    "cs_last_error",
    # placement layer (include/conserve_sched.h)
    "cs_prefill_curve_fit", "cs_prefill_curve_eval", "cs_provision_decoders",
    "cs_place_least_occupied", "cs_sched_create", "cs_sched_destroy", "cs_sched_admit",
    "cs_sched_bind",
]
PROFILE_KINDS = ["append", "pack", "unpack", "decode_split", "decode_merge", "attn_fwd", "mixed_layer"]


class ConserveError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class PoolDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_convs", ctypes.c_int32), ("max_pages_per_conv", ctypes.c_int32),
                ("n_pages", ctypes.c_int64)]


class DeviceInfo(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 256), ("arch", ctypes.c_char * 64),
                ("cu_count", ctypes.c_int32), ("clock_khz", ctypes.c_int32),
                ("memory_clock_khz", ctypes.c_int32), ("memory_bus_width_bits", ctypes.c_int32),
                ("lds_per_cu_bytes", ctypes.c_int64), ("lds_per_block_bytes", ctypes.c_int64),
                ("l2_bytes", ctypes.c_int64), ("total_mem_bytes", ctypes.c_int64)]


class PrefillCurve(ctypes.Structure):
    _fields_ = [("c0", ctypes.c_double), ("c1", ctypes.c_double), ("c2", ctypes.c_double)]


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
        "cs_attn_decode_batch_noalloc": (I32, [P, I32, PI32, I32, VP, VP, VP]),
        "cs_mixed_step": (I32, [P, I32, PI32, PI32, I32, PI32, VP, VP, VP, VP, VP, VP, ctypes.c_uint32, VP]),
        "cs_kv_pack_size": (I32, [P, I32, ctypes.POINTER(SZ)]),
        "cs_kv_pack": (I32, [P, I32, VP, SZ, VP]),
        "cs_kv_unpack": (I32, [P, VP, SZ, I64, PI32, VP]),
        "cs_profile_start": (I32, [P]),
        "cs_profile_stop": (I32, [P, ctypes.POINTER(ctypes.c_double), PI64]),
        "cs_device_info": (I32, [I32, ctypes.POINTER(DeviceInfo)]),
        "cs_debug_fail_launches": (I32, [P, I64]),
        "cs_probe_stream_read": (I32, [VP, SZ, VP, VP]),
        "cs_last_error": (ctypes.c_char_p, []),
        "cs_prefill_curve_fit": (I32, [I32, PI64, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(PrefillCurve), ctypes.POINTER(ctypes.c_double)]),
        "cs_prefill_curve_eval": (I32, [ctypes.POINTER(PrefillCurve), I64, ctypes.POINTER(ctypes.c_double)]),
        "cs_provision_decoders": (I32, [ctypes.c_double] * 6 + [ctypes.POINTER(ctypes.c_double)] * 3 + [PI32]),
        "cs_place_least_occupied": (I32, [I32, PI64, PI64, I64, PI32]),
        "cs_sched_create": (I32, [ctypes.POINTER(PrefillCurve), ctypes.c_double, I32, ctypes.POINTER(P),
                                  ctypes.POINTER(P)]),
        "cs_sched_destroy": (I32, [P]),
        "cs_sched_admit": (I32, [P, I64, ctypes.c_double, ctypes.POINTER(ctypes.c_double),
                                 ctypes.POINTER(ctypes.c_double)]),
        "cs_sched_bind": (I32, [P, I64, PI32]),
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
        """The pool as [n_layers][n_pages][n_kv_heads][2*16*head_dim] bf16 bits (int16 view); each
        block is the K part (head_dim/32 sub-blocks [16 tokens][32 dims]) then V^T[head_dim][16]."""
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
        return self._decode(self.lib.cs_attn_decode_batch, convs, layer, q, out)

    def attn_decode_batch_noalloc(self, convs, layer, q, out) -> torch.Tensor:
        """cs_attn_decode_batch_noalloc: the caller passes `out` (nothing is allocated)."""
        return self._decode(self.lib.cs_attn_decode_batch_noalloc, convs, layer, q, out)

    def _decode(self, fn, convs, layer, q, out):
        ca, cp = _i32_array(convs)
        shp = (ca.size, self.n_q_heads, self.head_dim)
        qptr = self._dev(q, "q", shp)
        if out is None:
            out = torch.empty(shp, dtype=torch.bfloat16, device=self.device)
        optr = self._dev(out, "out", shp)
        _check(fn(self._handle, ca.size, cp, layer, qptr, optr, _stream_handle(self.device)))
        return out

    def mixed_step(self, ext_convs, ext_lens, dec_convs, k, v, q_ext=None, q_dec=None,
                   out_ext=None, out_dec=None, layer_ordered=False):
        """One decoder step: extend chunks + one decoded token per decoding conversation, appended
        for every layer, then attention of every layer. With layer_ordered, layer l+1's attention
        starts only after layer l's (extend and decode of one layer still overlap), as in a model
        forward pass. Returns (out_ext, out_dec)."""
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
        flags = CS_MIXED_LAYER_ORDERED if layer_ordered else 0
        _check(self.lib.cs_mixed_step(self._handle, ea.size, ep, lp, nd, dp, kp, vp, qe, oe, qd, od,
                                      flags, _stream_handle(self.device)))
        return out_ext, out_dec

    # -- instrumentation -----------------------------------------------------------------------
    def debug_fail_launches(self, after: int) -> None:
        """cs_debug_fail_launches: launches after the next `after` report CS_EHIP (after < 0: off)."""
        _check(self.lib.cs_debug_fail_launches(self._handle, int(after)))

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


# ------------------------------------------------------------------------------------------------
# instrumentation
# ------------------------------------------------------------------------------------------------
def device_info(device: int = 0) -> dict:
    """cs_device_info: name, arch, CU count, clocks, LDS, L2 and memory size of a HIP device."""
    lib = load_library()
    d = DeviceInfo()
    _check(lib.cs_device_info(int(device), ctypes.byref(d)))
    out = {f: getattr(d, f) for f, _ in DeviceInfo._fields_}
    out["name"], out["arch"] = d.name.decode(), d.arch.decode()
    return out


def probe_stream_read(src: torch.Tensor, sink: torch.Tensor) -> None:
    """cs_probe_stream_read over a contiguous device tensor (its byte size rounded down to 16) on
    the current stream; sink: >= 4 bytes of device memory."""
    lib = load_library()
    if src.device.type != "cuda" or not src.is_contiguous() or sink.device.type != "cuda":
        raise ValueError("src and sink must be contiguous device tensors")
    nbytes = (src.numel() * src.element_size()) // 16 * 16
    _check(lib.cs_probe_stream_read(src.data_ptr(), nbytes, sink.data_ptr(),
                                    _stream_handle(src.device)))


# ------------------------------------------------------------------------------------------------
# placement layer (include/conserve_sched.h)
# ------------------------------------------------------------------------------------------------
def prefill_curve_fit(tokens, seconds):
    """Least-squares quadratic t(L) = c0 + c1 L + c2 L^2; returns ((c0, c1, c2), r2)."""
    lib = load_library()
    t = np.ascontiguousarray(np.asarray(tokens, dtype=np.int64).reshape(-1))
    y = np.ascontiguousarray(np.asarray(seconds, dtype=np.float64).reshape(-1))
    if t.size != y.size:
        raise ValueError("tokens and seconds differ in length")
    c, r2 = PrefillCurve(), ctypes.c_double()
    _check(lib.cs_prefill_curve_fit(int(t.size), t.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                    y.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                    ctypes.byref(c), ctypes.byref(r2)))
    return (c.c0, c.c1, c.c2), r2.value


def prefill_curve_eval(coef, tokens: int) -> float:
    lib = load_library()
    c, out = PrefillCurve(*coef), ctypes.c_double()
    _check(lib.cs_prefill_curve_eval(ctypes.byref(c), int(tokens), ctypes.byref(out)))
    return out.value


def provision_decoders(prefill_tokens_per_s, mean_turn1_tokens, decoder_tokens_per_s,
                       mean_decoder_tokens, convs_per_decoder, mean_lifetime_s):
    """Section 4.1 sizing; returns dict(saturation_rate, n_throughput, n_memory, n_decoders)."""
    lib = load_library()
    r, a, b = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    n = ctypes.c_int32()
    _check(lib.cs_provision_decoders(float(prefill_tokens_per_s), float(mean_turn1_tokens),
                                     float(decoder_tokens_per_s), float(mean_decoder_tokens),
                                     float(convs_per_decoder), float(mean_lifetime_s),
                                     ctypes.byref(r), ctypes.byref(a), ctypes.byref(b), ctypes.byref(n)))
    return {"saturation_rate": r.value, "n_throughput": a.value, "n_memory": b.value,
            "n_decoders": n.value}


def place_least_occupied(used_pages, free_pages, need_pages: int) -> int:
    """Index of the decoder the binding rule picks, or -1 (CS_ENOMEM) when none fits."""
    lib = load_library()
    u = np.ascontiguousarray(np.asarray(used_pages, dtype=np.int64).reshape(-1))
    f = np.ascontiguousarray(np.asarray(free_pages, dtype=np.int64).reshape(-1))
    if u.size != f.size:
        raise ValueError("used_pages and free_pages differ in length")
    d = ctypes.c_int32()
    code = lib.cs_place_least_occupied(int(u.size), u.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                       f.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                       int(need_pages), ctypes.byref(d))
    if code == CS_ENOMEM:
        return -1
    _check(code)
    return d.value


class Scheduler:
    """Reactive conversation placement over decoder KVPools (cs_sched_*). The pools stay owned
    by the caller and must outlive the scheduler."""

    def __init__(self, coef, max_wait_s: float, decoders=()):
        """decoders = () makes an admission-only scheduler (bind() then raises CS_EINVAL)."""
        self.lib = load_library()
        self.decoders = list(decoders)
        arr = (ctypes.c_void_p * max(1, len(self.decoders)))(*[d._handle for d in self.decoders])
        c = PrefillCurve(*coef)
        h = ctypes.c_void_p()
        _check(self.lib.cs_sched_create(ctypes.byref(c), float(max_wait_s), len(self.decoders),
                                        ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)),
                                        ctypes.byref(h)))
        self._handle = h

    def admit(self, turn1_tokens: int, now_s: float):
        """(start_s, done_s) of the turn-1 prefill, or None when refused (CS_EBUSY)."""
        a, b = ctypes.c_double(), ctypes.c_double()
        code = self.lib.cs_sched_admit(self._handle, int(turn1_tokens), float(now_s),
                                       ctypes.byref(a), ctypes.byref(b))
        if code == CS_EBUSY:
            return None
        _check(code)
        return a.value, b.value

    def bind(self, kv_tokens: int) -> int:
        """Decoder index for a conversation of kv_tokens tokens, or -1 (CS_ENOMEM)."""
        d = ctypes.c_int32()
        code = self.lib.cs_sched_bind(self._handle, int(kv_tokens), ctypes.byref(d))
        if code == CS_ENOMEM:
            return -1
        _check(code)
        return d.value

    def close(self) -> None:
        if self._handle:
            _check(self.lib.cs_sched_destroy(self._handle))
            self._handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
