"""Python binding of libdla (ctypes).  Argument marshalling only: every step of
the layer runs in the HIP kernels of libdla.so; torch provides device memory and
the current stream.  The library must be built (python -m
paper_2606_10650_amd.build); a missing library is an error, there is no
fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdla.so")
_lib = None

DLA_OK, DLA_ERR_INVALID_ARG, DLA_ERR_UNSUPPORTED, DLA_ERR_CACHE_MISMATCH, DLA_ERR_HIP, \
    DLA_ERR_WORKSPACE = range(6)
DLA_F32, DLA_BF16 = 0, 1
DLA_SKIP_READOUT = 1
DLA_SERIAL_STAGES = 2
DLA_POOL_BUDGET_SHIFT = 8  # flags bits 8..15: log2 of the state-copy budget in bytes
DLA_FLAG_BAD_MERGE_OVERRIDE = 1
DLA_FLAG_CACHE_MISMATCH = 2

EXPORTED = ("dla_cache_layout_of", "dla_state_cache_alloc", "dla_cache_flags",
            "dla_cache_header_check", "dla_prefill_workspace_size", "dla_prefill_segment_count",
            "dla_prefill_segment_starts", "dla_prefill", "dla_prefill_static", "dla_decode_step",
            "dla_decode_step_delta", "dla_prefill_delta_workspace_size", "dla_prefill_delta",
            "dla_status_string", "dla_get_last_error", "dla_peak_mfma_bf16", "dla_peak_hbm_read")
STATIC_SCRATCH_BYTES = 128 << 20   # DLA_STATIC_SCRATCH_BYTES


class CacheDesc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("C", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("state_dtype", ctypes.c_int32)]


class Params(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("eps", ctypes.c_float), ("eps_rms", ctypes.c_float),
                ("flags", ctypes.c_uint32), ("stage_events", ctypes.c_void_p),
                ("readout_events", ctypes.c_void_p), ("n_readout_events", ctypes.c_int32)]


PREFILL_STAGES = ("frames", "scan", "update", "readout")


class Layout(ctypes.Structure):
    _fields_ = [("meta_offset", ctypes.c_size_t), ("meta_stride", ctypes.c_size_t),
                ("states_offset", ctypes.c_size_t), ("open_offset", ctypes.c_size_t),
                ("total_bytes", ctypes.c_size_t)]


class DLAError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


def lib():
    """Load libdla.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_10650_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I = ctypes.c_int
        L.dla_cache_layout_of.argtypes = [ctypes.POINTER(CacheDesc), ctypes.POINTER(Layout)]
        L.dla_state_cache_alloc.argtypes = [ctypes.POINTER(CacheDesc), P,
                                            ctypes.POINTER(ctypes.c_size_t), P]
        L.dla_cache_flags.argtypes = [ctypes.POINTER(CacheDesc), P, ctypes.POINTER(ctypes.c_uint32),
                                      P]
        L.dla_cache_header_check.argtypes = [ctypes.POINTER(CacheDesc), P,
                                             ctypes.POINTER(ctypes.c_uint32)]
        L.dla_prefill_workspace_size.argtypes = [ctypes.POINTER(CacheDesc), ctypes.c_int32, I,
                                                 ctypes.c_uint32, ctypes.POINTER(ctypes.c_size_t)]
        L.dla_prefill_segment_count.argtypes = [ctypes.POINTER(CacheDesc), ctypes.c_int32, I,
                                                ctypes.c_uint32, ctypes.POINTER(ctypes.c_int32)]
        L.dla_prefill_segment_starts.argtypes = [ctypes.POINTER(CacheDesc), ctypes.c_int32, I,
                                                 ctypes.c_uint32, ctypes.POINTER(ctypes.c_int32),
                                                 ctypes.c_int32]
        L.dla_prefill.argtypes = [ctypes.POINTER(CacheDesc), P, P, P, P, P, P, ctypes.c_int32, I,
                                  ctypes.POINTER(Params), P, I, P, P, P, P, P, P, ctypes.c_size_t, P]
        L.dla_prefill_static.argtypes = [ctypes.POINTER(CacheDesc), P, P, P, P, P, P,
                                         ctypes.c_int32, I, ctypes.POINTER(Params), P, I, P, P, P,
                                         P, P, P]
        L.dla_decode_step.argtypes = [ctypes.POINTER(CacheDesc), P, P, P, P, P, P, I,
                                      ctypes.POINTER(Params), P, I, P, P, P, P, P, P]
        L.dla_decode_step_delta.argtypes = [ctypes.POINTER(CacheDesc), P, P, P, P, P, P, P, I,
                                            ctypes.POINTER(Params), P, I, P, P, P, P, P, P]
        L.dla_prefill_delta_workspace_size.argtypes = [ctypes.POINTER(CacheDesc), ctypes.c_int32,
                                                       I, ctypes.c_uint32,
                                                       ctypes.POINTER(ctypes.c_size_t)]
        L.dla_prefill_delta.argtypes = [ctypes.POINTER(CacheDesc), P, P, P, P, P, P, P,
                                        ctypes.c_int32, I, ctypes.POINTER(Params), P, I, P, P, P,
                                        P, P, P, ctypes.c_size_t, P]
        L.dla_peak_mfma_bf16.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P]
        L.dla_peak_hbm_read.argtypes = [P, ctypes.c_size_t, ctypes.c_int32, P, P]
        L.dla_status_string.argtypes = [I]
        L.dla_status_string.restype = ctypes.c_char_p
        L.dla_get_last_error.argtypes = []
        for name in ("dla_cache_layout_of", "dla_state_cache_alloc", "dla_cache_flags",
                     "dla_cache_header_check", "dla_prefill_workspace_size",
                     "dla_prefill_segment_count", "dla_prefill_segment_starts", "dla_prefill",
                     "dla_prefill_static", "dla_decode_step", "dla_decode_step_delta",
                     "dla_prefill_delta_workspace_size", "dla_prefill_delta", "dla_get_last_error",
                     "dla_peak_mfma_bf16", "dla_peak_hbm_read"):
            getattr(L, name).restype = I
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().dla_status_string(int(s)).decode()


def _check(status: int, what: str):
    if status != DLA_OK:
        raise DLAError(status, what)


def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t == torch.float32:
        return DLA_F32
    if t == torch.bfloat16:
        return DLA_BF16
    raise ValueError(f"unsupported dtype {t}")


def _ptr(t) -> Optional[int]:
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


@dataclasses.dataclass
class StateCache:
    """A device state cache (Sec. 3.2) for B*H heads of capacity C.  state_dtype
    is the storage type of the states (DLA_F32, or DLA_BF16: closed states in
    bfloat16, the newest state of each head in float32)."""
    B: int
    H: int
    C: int
    d_k: int
    d_v: int
    buf: "object"  # torch uint8 tensor on the device
    state_dtype: int = DLA_F32

    @property
    def desc(self) -> CacheDesc:
        return CacheDesc(self.B, self.H, self.C, self.d_k, self.d_v, self.state_dtype)

    @property
    def device(self):
        return self.buf.device


def cache_layout(B, H, C, d_k, d_v, state_dtype: int = DLA_F32) -> Layout:
    L = Layout()
    _check(lib().dla_cache_layout_of(ctypes.byref(CacheDesc(B, H, C, d_k, d_v, state_dtype)),
                                     ctypes.byref(L)), "dla_cache_layout_of")
    return L


def cache_alloc(B: int, H: int, C: int, d_k: int, d_v: int, device="cuda",
                state_dtype: int = DLA_F32) -> StateCache:
    """Allocate and initialise an empty cache (two-call dla_state_cache_alloc)."""
    torch = _torch()
    d = CacheDesc(B, H, C, d_k, d_v, state_dtype)
    n = ctypes.c_size_t(0)
    _check(lib().dla_state_cache_alloc(ctypes.byref(d), None, ctypes.byref(n), None),
           "dla_state_cache_alloc(size)")
    buf = torch.empty(n.value, dtype=torch.uint8, device=device)
    _check(lib().dla_state_cache_alloc(ctypes.byref(d), _ptr(buf), ctypes.byref(n),
                                       _stream(buf.device)), "dla_state_cache_alloc")
    return StateCache(B, H, C, d_k, d_v, buf, state_dtype)


def cache_reset(cache: StateCache) -> None:
    """Empty an allocated cache in place (dla_state_cache_alloc on its buffer)."""
    n = ctypes.c_size_t(cache.buf.numel())
    _check(lib().dla_state_cache_alloc(ctypes.byref(cache.desc), _ptr(cache.buf), ctypes.byref(n),
                                       _stream(cache.device)), "dla_state_cache_alloc")


def header_check(desc: CacheDesc, header: bytes) -> int:
    """dla_cache_header_check on a host copy of a cache header: the device
    flags, or DLAError (DLA_ERR_CACHE_MISMATCH) when it does not match desc."""
    f = ctypes.c_uint32(0)
    buf = ctypes.create_string_buffer(bytes(header), len(header))
    _check(lib().dla_cache_header_check(ctypes.byref(desc), buf, ctypes.byref(f)),
           "dla_cache_header_check")
    return int(f.value)


def cache_flags(cache: StateCache) -> int:
    f = ctypes.c_uint32(0)
    _check(lib().dla_cache_flags(ctypes.byref(cache.desc), _ptr(cache.buf), ctypes.byref(f),
                                 _stream(cache.device)), "dla_cache_flags")
    return int(f.value)


def _flags(skip_readout: bool, serial: bool, pool_budget_log2: int = 0) -> int:
    """params flags; pool_budget_log2: DLA_POOL_BUDGET_LOG2 (0: the default budget)."""
    return ((DLA_SKIP_READOUT if skip_readout else 0) | (DLA_SERIAL_STAGES if serial else 0) |
            ((int(pool_budget_log2) & 0xFF) << DLA_POOL_BUDGET_SHIFT))


def workspace_bytes(cache: StateCache, T: int, dtype=None, skip_readout: bool = False,
                    serial: bool = False, pool_budget_log2: int = 0) -> int:
    """Prefill workspace for T tokens of input dtype (torch dtype, default bf16)."""
    code = DLA_BF16 if dtype is None else _dtype_code(dtype)
    n = ctypes.c_size_t(0)
    _check(lib().dla_prefill_workspace_size(ctypes.byref(cache.desc), int(T), code,
                                            _flags(skip_readout, serial, pool_budget_log2),
                                            ctypes.byref(n)), "dla_prefill_workspace_size")
    return int(n.value)


def delta_workspace_bytes(cache: StateCache, T: int, dtype=None, skip_readout: bool = False,
                          pool_budget_log2: int = 0, serial: bool = False) -> int:
    """dla_prefill_delta workspace for T tokens of input dtype (default bf16)."""
    code = DLA_BF16 if dtype is None else _dtype_code(dtype)
    n = ctypes.c_size_t(0)
    _check(lib().dla_prefill_delta_workspace_size(ctypes.byref(cache.desc), int(T), code,
                                                  _flags(skip_readout, serial, pool_budget_log2),
                                                  ctypes.byref(n)),
           "dla_prefill_delta_workspace_size")
    return int(n.value)


def prefill_segments(cache: StateCache, T: int, dtype=None, skip_readout: bool = False,
                     serial: bool = False, pool_budget_log2: int = 0) -> int:
    """Segments (readout launches) of a prefill of T tokens."""
    code = DLA_BF16 if dtype is None else _dtype_code(dtype)
    n = ctypes.c_int32(0)
    _check(lib().dla_prefill_segment_count(ctypes.byref(cache.desc), int(T), code,
                                           _flags(skip_readout, serial, pool_budget_log2), ctypes.byref(n)),
           "dla_prefill_segment_count")
    return int(n.value)


def prefill_segment_starts(cache: StateCache, T: int, dtype=None, skip_readout: bool = False,
                           serial: bool = False, pool_budget_log2: int = 0) -> list:
    """First token of each segment of a prefill of T tokens."""
    code = DLA_BF16 if dtype is None else _dtype_code(dtype)
    n = prefill_segments(cache, T, dtype, skip_readout, serial, pool_budget_log2)
    arr = (ctypes.c_int32 * n)()
    _check(lib().dla_prefill_segment_starts(ctypes.byref(cache.desc), int(T), code,
                                            _flags(skip_readout, serial, pool_budget_log2), arr, n),
           "dla_prefill_segment_starts")
    return list(arr)


def _event_array(events):
    # torch.cuda.Event objects (enable_timing=True)
    return (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])


def _params(tau, eps, eps_rms, skip_readout, serial=False, stage_events=None,
            readout_events=None, pool_budget_log2=0):
    p = Params(float(tau), float(eps), float(eps_rms),
               _flags(skip_readout, serial, pool_budget_log2), None, None, 0)
    keep = []
    if stage_events is not None:
        assert len(stage_events) == len(PREFILL_STAGES) + 1
        arr = _event_array(stage_events)
        keep.append(arr)
        p.stage_events = ctypes.cast(arr, ctypes.c_void_p)
    if readout_events:
        arr = _event_array(readout_events)
        keep.append(arr)
        p.readout_events = ctypes.cast(arr, ctypes.c_void_p)
        p.n_readout_events = len(readout_events)
    p._events_keepalive = keep  # the arrays must outlive the call
    return p


def prefill(cache: StateCache, q, k, v, g, lam=None, *, tau: float = 0.5, eps: float = 1e-6,
            eps_rms: float = 1e-6, out=None, out_dtype=None, skip_readout: bool = False,
            boundary=None, merge_idx=None, score=None, boundary_override=None,
            merge_override=None, workspace=None, want_exports: bool = True, stage_events=None,
            serial: bool = False, readout_events=None, pool_budget_log2: int = 0):
    """Absorb T tokens per head.  q, k: [B, H, T, d_k]; v: [B, H, T, d_v]; g:
    [B, H, T] float32; lam: [B, H, T, C] or None.  serial: run the stages one
    after another on the current stream (otherwise the scan of long inputs is
    overlapped with the later stages on a second stream).  pool_budget_log2:
    log2 of the bytes of state copies per call (0: the library's default).
    Returns (out, boundary, merge_idx, score); exports not requested are None."""
    torch = _torch()
    B, H, C = cache.B, cache.H, cache.C
    T = k.shape[2]
    dev = cache.device
    assert k.shape == (B, H, T, cache.d_k) and v.shape == (B, H, T, cache.d_v), (k.shape, v.shape)
    assert g.shape == (B, H, T) and g.dtype == torch.float32
    for t in (q, k, v, g, lam, boundary_override, merge_override):
        assert t is None or (t.is_contiguous() and t.device == dev)
    if q is not None:
        assert q.shape == (B, H, T, cache.d_k) and q.dtype == k.dtype
    if lam is not None:
        assert lam.shape == (B, H, T, C) and lam.dtype == k.dtype
    if out is None and not skip_readout:
        out = torch.empty((B, H, T, cache.d_v), dtype=out_dtype or k.dtype, device=dev)
    if want_exports:
        boundary = boundary if boundary is not None else torch.empty((B, H, T), dtype=torch.int8,
                                                                      device=dev)
        merge_idx = merge_idx if merge_idx is not None else torch.empty((B, H, T),
                                                                        dtype=torch.int32,
                                                                        device=dev)
        score = score if score is not None else torch.empty((B, H, T), dtype=torch.float32,
                                                            device=dev)
    wsb = workspace_bytes(cache, T, k.dtype, skip_readout, serial, pool_budget_log2)
    if workspace is None or workspace.numel() < wsb:
        workspace = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
    for e in list(stage_events or ()) + list(readout_events or ()):
        if not e.cuda_event:
            e.record()   # torch creates an event on its first record
    p = _params(tau, eps, eps_rms, skip_readout, serial, stage_events, readout_events,
                pool_budget_log2)
    st = lib().dla_prefill(ctypes.byref(cache.desc), _ptr(cache.buf), _ptr(q), _ptr(k), _ptr(v),
                           _ptr(g), _ptr(lam), int(T), _dtype_code(k.dtype), ctypes.byref(p),
                           _ptr(out), _dtype_code(out.dtype) if out is not None else DLA_F32,
                           _ptr(boundary), _ptr(merge_idx), _ptr(score), _ptr(boundary_override),
                           _ptr(merge_override), _ptr(workspace), workspace.numel(),
                           _stream(dev))
    _check(st, "dla_prefill")
    return out, boundary, merge_idx, score


def prefill_static(cache: StateCache, q, k, v, g, lam=None, *, tau: float = 0.5,
                   eps: float = 1e-6, eps_rms: float = 1e-6, out, boundary=None, merge_idx=None,
                   score=None, boundary_override=None, merge_override=None,
                   skip_readout: bool = False, pool_budget_log2: int = 0):
    """dla_prefill_static: prefill with the library's static device scratch as
    workspace (stages serial).  Allocates nothing: the caller passes the output
    and any export buffers.  Shapes as prefill."""
    B, H, C = cache.B, cache.H, cache.C
    T = k.shape[2]
    dev = cache.device
    assert k.shape == (B, H, T, cache.d_k) and v.shape == (B, H, T, cache.d_v)
    assert g.shape == (B, H, T)
    for t in (q, k, v, g, lam, out, boundary, merge_idx, score, boundary_override,
              merge_override):
        assert t is None or (t.is_contiguous() and t.device == dev)
    p = _params(tau, eps, eps_rms, skip_readout, serial=True, pool_budget_log2=pool_budget_log2)
    st = lib().dla_prefill_static(ctypes.byref(cache.desc), _ptr(cache.buf), _ptr(q), _ptr(k),
                                  _ptr(v), _ptr(g), _ptr(lam), int(T), _dtype_code(k.dtype),
                                  ctypes.byref(p), _ptr(out),
                                  _dtype_code(out.dtype) if out is not None else DLA_F32,
                                  _ptr(boundary), _ptr(merge_idx), _ptr(score),
                                  _ptr(boundary_override), _ptr(merge_override), _stream(dev))
    _check(st, "dla_prefill_static")
    return out, boundary, merge_idx, score


def decode_step(cache: StateCache, q, k, v, g, lam=None, *, tau: float = 0.5, eps: float = 1e-6,
                eps_rms: float = 1e-6, out=None, out_dtype=None, skip_readout: bool = False,
                boundary=None, merge_idx=None, score=None, boundary_override=None,
                merge_override=None, want_exports: bool = True):
    """Absorb one token per head.  q, k: [B, H, d_k]; v: [B, H, d_v]; g: [B, H];
    lam: [B, H, C] or None."""
    torch = _torch()
    B, H, C = cache.B, cache.H, cache.C
    dev = cache.device
    assert k.shape == (B, H, cache.d_k) and v.shape == (B, H, cache.d_v)
    assert g.shape == (B, H) and g.dtype == torch.float32
    for t in (q, k, v, g, lam, boundary_override, merge_override):
        assert t is None or (t.is_contiguous() and t.device == dev)
    if lam is not None:
        assert lam.shape == (B, H, C) and lam.dtype == k.dtype
    if out is None and not skip_readout:
        out = torch.empty((B, H, cache.d_v), dtype=out_dtype or k.dtype, device=dev)
    if want_exports:
        boundary = boundary if boundary is not None else torch.empty((B, H), dtype=torch.int8,
                                                                      device=dev)
        merge_idx = merge_idx if merge_idx is not None else torch.empty((B, H), dtype=torch.int32,
                                                                        device=dev)
        score = score if score is not None else torch.empty((B, H), dtype=torch.float32,
                                                            device=dev)
    p = _params(tau, eps, eps_rms, skip_readout)
    st = lib().dla_decode_step(ctypes.byref(cache.desc), _ptr(cache.buf), _ptr(q), _ptr(k),
                               _ptr(v), _ptr(g), _ptr(lam), _dtype_code(k.dtype), ctypes.byref(p),
                               _ptr(out), _dtype_code(out.dtype) if out is not None else DLA_F32,
                               _ptr(boundary), _ptr(merge_idx), _ptr(score),
                               _ptr(boundary_override), _ptr(merge_override), _stream(dev))
    _check(st, "dla_decode_step")
    return out, boundary, merge_idx, score


def decode_step_delta(cache: StateCache, q, k, v, g, beta, lam=None, *, tau: float = 0.5,
                      eps: float = 1e-6, eps_rms: float = 1e-6, out=None, out_dtype=None,
                      skip_readout: bool = False, boundary=None, merge_idx=None, score=None,
                      boundary_override=None, merge_override=None, want_exports: bool = True):
    """dla_decode_step_delta: one token per head in the Gated DeltaNet form.
    Shapes as decode_step; beta: [B, H] float32 step sizes."""
    torch = _torch()
    B, H = cache.B, cache.H
    dev = cache.device
    assert beta is not None and beta.shape == (B, H) and beta.dtype == torch.float32
    assert k.shape == (B, H, cache.d_k) and v.shape == (B, H, cache.d_v) and g.shape == (B, H)
    for t in (q, k, v, g, beta, lam, boundary_override, merge_override):
        assert t is None or (t.is_contiguous() and t.device == dev)
    if out is None and not skip_readout:
        out = torch.empty((B, H, cache.d_v), dtype=out_dtype or k.dtype, device=dev)
    if want_exports:
        boundary = boundary if boundary is not None else torch.empty((B, H), dtype=torch.int8,
                                                                      device=dev)
        merge_idx = merge_idx if merge_idx is not None else torch.empty((B, H), dtype=torch.int32,
                                                                        device=dev)
        score = score if score is not None else torch.empty((B, H), dtype=torch.float32,
                                                            device=dev)
    p = _params(tau, eps, eps_rms, skip_readout)
    st = lib().dla_decode_step_delta(ctypes.byref(cache.desc), _ptr(cache.buf), _ptr(q), _ptr(k),
                                     _ptr(v), _ptr(g), _ptr(beta), _ptr(lam), _dtype_code(k.dtype),
                                     ctypes.byref(p), _ptr(out),
                                     _dtype_code(out.dtype) if out is not None else DLA_F32,
                                     _ptr(boundary), _ptr(merge_idx), _ptr(score),
                                     _ptr(boundary_override), _ptr(merge_override), _stream(dev))
    _check(st, "dla_decode_step_delta")
    return out, boundary, merge_idx, score


def prefill_delta(cache: StateCache, q, k, v, g, beta, lam=None, *, tau: float = 0.5,
                  eps: float = 1e-6, eps_rms: float = 1e-6, out=None, out_dtype=None,
                  skip_readout: bool = False, boundary=None, merge_idx=None, score=None,
                  boundary_override=None, merge_override=None, workspace=None,
                  want_exports: bool = True, pool_budget_log2: int = 0, serial: bool = False):
    """dla_prefill_delta: T tokens per head in the Gated DeltaNet form.  Shapes
    as prefill; beta: [B, H, T] float32; serial: DLA_SERIAL_STAGES.  The
    workspace is allocated when none (or one too small) is given."""
    torch = _torch()
    B, H, C = cache.B, cache.H, cache.C
    T = k.shape[2]
    dev = cache.device
    assert k.shape == (B, H, T, cache.d_k) and v.shape == (B, H, T, cache.d_v)
    assert g.shape == (B, H, T) and beta is not None and beta.shape == (B, H, T)
    assert beta.dtype == torch.float32
    for t in (q, k, v, g, beta, lam, boundary_override, merge_override):
        assert t is None or (t.is_contiguous() and t.device == dev)
    if lam is not None:
        assert lam.shape == (B, H, T, C) and lam.dtype == k.dtype
    if out is None and not skip_readout:
        out = torch.empty((B, H, T, cache.d_v), dtype=out_dtype or k.dtype, device=dev)
    if want_exports:
        boundary = boundary if boundary is not None else torch.empty((B, H, T), dtype=torch.int8,
                                                                      device=dev)
        merge_idx = merge_idx if merge_idx is not None else torch.empty((B, H, T),
                                                                        dtype=torch.int32,
                                                                        device=dev)
        score = score if score is not None else torch.empty((B, H, T), dtype=torch.float32,
                                                            device=dev)
    wsb = delta_workspace_bytes(cache, T, k.dtype, skip_readout, pool_budget_log2, serial)
    if workspace is None or workspace.numel() < wsb:
        workspace = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
    p = _params(tau, eps, eps_rms, skip_readout, serial=serial, pool_budget_log2=pool_budget_log2)
    st = lib().dla_prefill_delta(ctypes.byref(cache.desc), _ptr(cache.buf), _ptr(q), _ptr(k),
                                 _ptr(v), _ptr(g), _ptr(beta), _ptr(lam), int(T),
                                 _dtype_code(k.dtype), ctypes.byref(p), _ptr(out),
                                 _dtype_code(out.dtype) if out is not None else DLA_F32,
                                 _ptr(boundary), _ptr(merge_idx), _ptr(score),
                                 _ptr(boundary_override), _ptr(merge_override), _ptr(workspace),
                                 workspace.numel(), _stream(dev))
    _check(st, "dla_prefill_delta")
    return out, boundary, merge_idx, score


def cache_export(cache: StateCache, heads=None) -> dict:
    """Read a cache back to host memory and decode its byte layout (dla.h): per
    head m, G, tokens, and in chronological order F, Ibar, n, perm, and the
    stored values of each state as float64 [n_heads, C, d_k, d_v] (entries
    j >= m are zero).  Stored values are in the state's own frame: the true
    state is exp(G - F[j]) times them (lazy decay).  With bfloat16 storage the
    newest state's values come from the float32 open region.  Only the bytes of
    the requested heads are copied."""
    sd = cache.state_dtype
    L = cache_layout(cache.B, cache.H, cache.C, cache.d_k, cache.d_v, sd)
    nh = cache.B * cache.H
    heads = list(range(nh)) if heads is None else list(heads)
    C, dk, dv = cache.C, cache.d_k, cache.d_v
    D = dk * dv
    es = 2 if sd == DLA_BF16 else 4
    buf = cache.buf

    def host(a, b):
        return buf[a:b].cpu().numpy()

    hdr = host(0, 256)
    res = {"m": np.zeros(len(heads), np.int32), "G": np.zeros(len(heads)),
           "tokens": np.zeros(len(heads), np.int64), "F": np.zeros((len(heads), C)),
           "ibar": np.zeros((len(heads), C)), "n": np.zeros((len(heads), C), np.int32),
           "perm": np.zeros((len(heads), C), np.int32),
           "stored": np.zeros((len(heads), C, dk, dv)),
           "flags": int(hdr[28:32].view(np.uint32)[0])}
    for i, h in enumerate(heads):
        base = L.meta_offset + h * L.meta_stride
        mb = host(base, base + L.meta_stride)
        m = int(mb[0:4].view(np.int32)[0])
        res["m"][i] = m
        res["G"][i] = mb[8:16].view(np.float64)[0]
        res["tokens"][i] = mb[16:24].view(np.int64)[0]
        res["F"][i] = mb[32:32 + 8 * C].view(np.float64)
        res["ibar"][i] = mb[32 + 8 * C:32 + 16 * C].view(np.float64)
        res["n"][i] = mb[32 + 16 * C:32 + 20 * C].view(np.int32)
        perm = mb[32 + 20 * C:32 + 24 * C].view(np.int32)
        res["perm"][i] = perm
        s0 = L.states_offset + h * C * D * es
        raw = host(s0, s0 + C * D * es)
        if sd == DLA_BF16:
            slots = (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32)
        else:
            slots = raw.view(np.float32)
        slots = slots.reshape(C, dk, dv)
        # (with bfloat16 storage the newest state lives in the float32 open
        # region, and its slot holds nothing)
        for j in range(m - 1 if sd == DLA_BF16 else m):
            res["stored"][i, j] = slots[perm[j]]
        if sd == DLA_BF16 and m > 0:
            o0 = L.open_offset + h * D * 4
            res["stored"][i, m - 1] = host(o0, o0 + D * 4).view(np.float32).reshape(dk, dv)
    return res


def peak_mfma_bf16(blocks: int, iters: int, sink) -> None:
    """Enqueue the dense bfloat16 MFMA rate kernel (blocks * 16 * iters * 32768
    operations); sink: a float32 device tensor of blocks * 256 elements."""
    assert sink.numel() >= blocks * 256
    _check(lib().dla_peak_mfma_bf16(int(blocks), int(iters), _ptr(sink), _stream(sink.device)),
           "dla_peak_mfma_bf16")


def peak_hbm_read(buf, blocks: int, sink) -> None:
    """Enqueue one read of the device buffer buf (bytes a multiple of 4096)."""
    assert sink.numel() >= blocks * 256
    nbytes = buf.numel() * buf.element_size()
    _check(lib().dla_peak_hbm_read(_ptr(buf), nbytes, int(blocks), _ptr(sink),
                                   _stream(sink.device)), "dla_peak_hbm_read")
