"""Python binding of the SAEF HIP library (``libsaef.so``).

Argument marshalling only: every function passes device pointers of torch
tensors, sizes and the current HIP stream to the C entry point of the same
name declared in ``include/saef.h`` and raises ``SaefError`` on a non-zero
return code.  Every step of the computation runs in the library's kernels.

Importing this module loads the library and raises ImportError when it has
not been built (``python -c "import __graft_entry__ as g; g.build()"``).
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# SAEF_LIBRARY may name another build of the library (e.g. a tuning variant)
LIB_PATH = os.environ.get("SAEF_LIBRARY") or os.path.join(HERE, "libsaef.so")

OK, EINVAL, ERANGE, EHIP = 0, -1, -2, -3
MODE_SC, MODE_DC = 0, 1
VARIANT_EF, VARIANT_SAEF = 0, 1

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build the HIP library first "
                      "(__graft_entry__.build())")

_lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.c_void_p
_i32, _i64, _f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float

_SIGS = {
    "saef_layout_create": [_P, _P, _i32, _i64, _i32, ctypes.POINTER(_P)],
    "saef_layout_destroy": [_P],
    "saef_layout_info": [_P, _P, _P, _P, _P],
    "saef_compress": [_P, _i32, _f32, _P, _P, _P, _P, _P],
    "saef_compress_momentum": [_P, _i32, _f32, _f32, _P, _P, _P, _P, _P, _P],
    "saef_aggregate": [_P, _i32, _i32, _P, _P, _P, _P, _P, _P, _P, _P],
    "saef_step_ahead": [_P, _i32, _P, _P, _P, _P],
    "saef_error_average": [_P, _i32, _P, _P],
    "saef_round": [_P, _i64, _i64, _i32, _f32, _i32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "saef_round_noalloc": [_P, _i64, _i64, _i32, _f32, _i32, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                           _P],
    "saef_round_momentum": [_P, _i64, _i64, _i32, _f32, _f32, _i32, _P, _P, _P, _P, _P, _P, _P,
                            _P, _P, _P, _P],
    "saef_round_begin": [_P, _i64, _i64, _i32, _i32, _i32, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                         _P],
    "saef_round_end": [_P, _i64, _i64, _i32, _f32, _f32, _i32, _P, _P, _P, _P, _P, _P, _P, _P,
                       _P, _P],
    "saef_topk_create": [_P, _P, ctypes.POINTER(_P)],
    "saef_topk_destroy": [_P],
    "saef_topk_info": [_P, _P],
    "saef_topk_compress": [_P, _i32, _f32, _f32, _P, _P, _P, _P, _P, _P, _P],
    "saef_topk_aggregate": [_P, _i32, _i32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "saef_topk_round": [_P, _i64, _i64, _i32, _f32, _f32, _i32, _P, _P, _P, _P, _P, _P, _P, _P,
                        _P, _P, _P, _P, _P],
    "saef_topk_round_begin": [_P, _i64, _i64, _i32, _i32, _i32, _P, _P, _P, _P, _P, _P, _P],
    "saef_topk_round_end": [_P, _i64, _i64, _i32, _f32, _f32, _i32, _P, _P, _P, _P, _P, _P, _P,
                            _P, _P, _P, _P, _P],
    "saef_topk_materialize": [_P, _i32, _P, _P, _P],
    "saef_materialize": [_P, _i32, _i32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "saef_status": [_P, _P],
    "saef_profile_enable": [_P, _i32, ctypes.c_uint32, _i32],
    "saef_profile_read": [_P, _P, _P],
    "saef_stream_probe": [_P, _P, _P, _i64, _P],
}
for _name, _args in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = ctypes.c_int

EXPORTS = tuple(_SIGS)

# kernel kinds of saef_profile_enable / saef_profile_read, in bit order
PROFILE_KINDS = ("step_ahead", "compress", "worker_scales", "aggregate", "server_scales",
                 "step_ahead_averaging", "mismatch")


class SaefError(RuntimeError):
    def __init__(self, fn: str, rc: int):
        names = {EINVAL: "SAEF_EINVAL", ERANGE: "SAEF_ERANGE", EHIP: "SAEF_EHIP"}
        super().__init__(f"{fn} returned {names.get(rc, rc)}")
        self.rc = rc


def _check(fn: str, rc: int) -> None:
    if rc != OK:
        raise SaefError(fn, rc)


def _dev(t, dtype):
    """Device pointer of a contiguous CUDA/HIP tensor of the given dtype (or None)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("SAEF buffers must be device tensors")
    if t.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError("SAEF buffers must be contiguous")
    return t.data_ptr()


def _f(t):
    return _dev(t, torch.float32)


def _w(t):
    if t is None:
        return None
    if t.dtype not in (torch.int64, torch.uint64):
        raise TypeError(f"sign words must be int64/uint64, got {t.dtype}")
    return _dev(t, t.dtype)


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


class Layout:
    """A tensor layout on the current device (see saef_layout_create)."""

    def __init__(self, offsets, sizes, d_pad: int, k_max: int):
        off = (ctypes.c_int64 * len(offsets))(*[int(v) for v in offsets])
        n = (ctypes.c_int64 * len(sizes))(*[int(v) for v in sizes])
        if len(off) != len(n):
            raise ValueError("offsets and sizes differ in length")
        handle = _P()
        _check("saef_layout_create",
               _lib.saef_layout_create(off, n, len(off), int(d_pad), int(k_max),
                                       ctypes.byref(handle)))
        self._h = handle
        self.L = len(off)
        self.d_pad = int(d_pad)
        self.k_max = int(k_max)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("layout destroyed")
        return self._h

    def info(self) -> dict:
        L, d, k, t = _i32(), _i64(), _i32(), _i64()
        _check("saef_layout_info", _lib.saef_layout_info(self.handle, ctypes.byref(L),
                                                         ctypes.byref(d), ctypes.byref(k),
                                                         ctypes.byref(t)))
        return {"L": L.value, "d_pad": d.value, "k_max": k.value, "n_tiles": t.value}

    def close(self) -> None:
        if getattr(self, "_h", None) is not None:
            _lib.saef_layout_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def saef_compress(layout: Layout, K: int, lr: float, g, e, signs, scales, stream=None):
    _check("saef_compress", _lib.saef_compress(layout.handle, K, lr, _f(g), _f(e), _w(signs),
                                               _f(scales), _stream(stream)))


def saef_compress_momentum(layout: Layout, K: int, lr: float, mu: float, g, m, e, signs, scales,
                           stream=None):
    _check("saef_compress_momentum",
           _lib.saef_compress_momentum(layout.handle, K, lr, mu, _f(g), _f(m), _f(e), _w(signs),
                                       _f(scales), _stream(stream)))


def saef_aggregate(layout: Layout, K: int, mode: int, signs, scales, x, e_srv=None,
                   srv_signs=None, srv_scales=None, avg=None, stream=None):
    _check("saef_aggregate", _lib.saef_aggregate(layout.handle, K, mode, _w(signs), _f(scales),
                                                 _f(avg), _f(e_srv), _w(srv_signs),
                                                 _f(srv_scales), _f(x), _stream(stream)))


def saef_step_ahead(layout: Layout, K: int, x, e, xh, stream=None):
    _check("saef_step_ahead", _lib.saef_step_ahead(layout.handle, K, _f(x), _f(e), _f(xh),
                                                   _stream(stream)))


def saef_error_average(layout: Layout, K: int, e, stream=None):
    _check("saef_error_average", _lib.saef_error_average(layout.handle, K, _f(e),
                                                         _stream(stream)))


def saef_round(layout: Layout, t: int, period: int, K: int, lr: float, mode: int, g, e, e_srv,
               x, xh, signs, scales, srv_signs=None, srv_scales=None, stream=None):
    _check("saef_round", _lib.saef_round(layout.handle, t, period, K, lr, mode, _f(g), _f(e),
                                         _f(e_srv), _f(x), _f(xh), _w(signs), _f(scales),
                                         _w(srv_signs), _f(srv_scales), _stream(stream)))


def saef_round_noalloc(layout: Layout, t: int, period: int, K: int, lr: float, mode: int, g, e,
                       e_srv, x, xh, signs, scales, srv_signs=None, srv_scales=None,
                       stream=None):
    _check("saef_round_noalloc",
           _lib.saef_round_noalloc(layout.handle, t, period, K, lr, mode, _f(g), _f(e), _f(e_srv),
                                   _f(x), _f(xh), _w(signs), _f(scales), _w(srv_signs),
                                   _f(srv_scales), _stream(stream)))


def saef_round_momentum(layout: Layout, t: int, period: int, K: int, lr: float, mu: float,
                        mode: int, g, m, e, e_srv, x, xh, signs, scales, srv_signs=None,
                        srv_scales=None, stream=None):
    _check("saef_round_momentum",
           _lib.saef_round_momentum(layout.handle, t, period, K, lr, mu, mode, _f(g), _f(m),
                                    _f(e), _f(e_srv), _f(x), _f(xh), _w(signs), _f(scales),
                                    _w(srv_signs), _f(srv_scales), _stream(stream)))


def _u32(t):
    """Rank words: int32 or uint32 device tensors (the same bits)."""
    if t is None:
        return None
    if t.dtype not in (torch.int32, torch.uint32):
        raise TypeError(f"rank words must be int32/uint32, got {t.dtype}")
    return _dev(t, t.dtype)


class TopK:
    """A Top-K plan on a layout (see saef_topk_create); keep[l] per tensor."""

    def __init__(self, layout: "Layout", keep):
        k = (ctypes.c_int64 * len(keep))(*[int(v) for v in keep])
        if len(k) != layout.L:
            raise ValueError("one kept count per tensor")
        handle = _P()
        _check("saef_topk_create", _lib.saef_topk_create(layout.handle, k, ctypes.byref(handle)))
        self._h = handle
        self.layout = layout  # the layout must outlive the plan
        total = _i64()
        _check("saef_topk_info", _lib.saef_topk_info(self._h, ctypes.byref(total)))
        self.total = int(total.value)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("plan destroyed")
        return self._h

    def destroy(self):
        if self._h is not None:
            _check("saef_topk_destroy", _lib.saef_topk_destroy(self._h))
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def saef_topk_compress(plan: TopK, K: int, lr: float, mu: float, g, m, e, sel, rank, vals,
                       stream=None):
    _check("saef_topk_compress",
           _lib.saef_topk_compress(plan.handle, K, lr, mu, _f(g), _f(m), _f(e), _w(sel),
                                   _u32(rank), _f(vals), _stream(stream)))


def saef_topk_aggregate(plan: TopK, K: int, mode: int, sel, rank, vals, x, e_srv=None,
                        srv_sel=None, srv_rank=None, srv_vals=None, avg=None, stream=None):
    _check("saef_topk_aggregate",
           _lib.saef_topk_aggregate(plan.handle, K, mode, _w(sel), _u32(rank), _f(vals), _f(avg),
                                    _f(e_srv), _w(srv_sel), _u32(srv_rank), _f(srv_vals), _f(x),
                                    _stream(stream)))


def saef_topk_round(plan: TopK, t: int, period: int, K: int, lr: float, mu: float, mode: int,
                    g, m, e, e_srv, x, xh, sel, rank, vals, srv_sel=None, srv_rank=None,
                    srv_vals=None, stream=None):
    _check("saef_topk_round",
           _lib.saef_topk_round(plan.handle, t, period, K, lr, mu, mode, _f(g), _f(m), _f(e),
                                _f(e_srv), _f(x), _f(xh), _w(sel), _u32(rank), _f(vals),
                                _w(srv_sel), _u32(srv_rank), _f(srv_vals), _stream(stream)))


def saef_topk_round_begin(plan: TopK, t: int, period: int, K: int, mode: int, variant: int, e,
                          sel, e_srv, x, xh, mismatch=None, stream=None):
    """First half of iteration t; sel: the selection words of the previous
    iteration (None only at t = 0)."""
    _check("saef_topk_round_begin",
           _lib.saef_topk_round_begin(plan.handle, t, period, K, mode, variant, _f(e), _w(sel),
                                      _f(e_srv), _f(x), _f(xh), _dev(mismatch, torch.float64),
                                      _stream(stream)))


def saef_topk_round_end(plan: TopK, t: int, period: int, K: int, lr: float, mu: float, mode: int,
                        g, m, e, e_srv, x, sel, rank, vals, srv_sel=None, srv_rank=None,
                        srv_vals=None, stream=None):
    """Second half of iteration t (the same t and period as the first)."""
    _check("saef_topk_round_end",
           _lib.saef_topk_round_end(plan.handle, t, period, K, lr, mu, mode, _f(g), _f(m), _f(e),
                                    _f(e_srv), _f(x), _w(sel), _u32(rank), _f(vals), _w(srv_sel),
                                    _u32(srv_rank), _f(srv_vals), _stream(stream)))


def saef_topk_materialize(plan: TopK, K: int, e, sel, stream=None):
    """The plain worker errors: e (K, d_pad) with the elements whose bit in
    sel is set put to 0, in place."""
    _check("saef_topk_materialize",
           _lib.saef_topk_materialize(plan.handle, K, _f(e), _w(sel), _stream(stream)))


def saef_round_begin(layout: Layout, t: int, period: int, K: int, mode: int, variant: int, e,
                     e_srv, x, xh, signs, scales, srv_signs=None, srv_scales=None,
                     mismatch=None, stream=None):
    """First half of iteration t; mismatch: float64 device tensor of 2 L or None."""
    _check("saef_round_begin",
           _lib.saef_round_begin(layout.handle, t, period, K, mode, variant, _f(e), _f(e_srv),
                                 _f(x), _f(xh), _w(signs), _f(scales), _w(srv_signs),
                                 _f(srv_scales), _dev(mismatch, torch.float64),
                                 _stream(stream)))


def saef_round_end(layout: Layout, t: int, period: int, K: int, lr: float, mu: float, mode: int,
                   g, m, e, e_srv, x, signs, scales, srv_signs=None, srv_scales=None,
                   stream=None):
    """Second half of iteration t (m None: no momentum, mu must be 0)."""
    _check("saef_round_end",
           _lib.saef_round_end(layout.handle, t, period, K, lr, mu, mode, _f(g), _f(m), _f(e),
                               _f(e_srv), _f(x), _w(signs), _f(scales), _w(srv_signs),
                               _f(srv_scales), _stream(stream)))


def saef_materialize(layout: Layout, K: int, mode: int, e, e_srv, x, signs, scales,
                     srv_signs=None, srv_scales=None, e_out=None, e_srv_out=None, x_out=None,
                     stream=None):
    _check("saef_materialize",
           _lib.saef_materialize(layout.handle, K, mode, _f(e), _f(e_srv), _f(x), _w(signs),
                                 _f(scales), _w(srv_signs), _f(srv_scales), _f(e_out),
                                 _f(e_srv_out), _f(x_out), _stream(stream)))


def saef_status(layout: Layout, stream=None) -> int:
    """SAEF_OK or SAEF_ERANGE (sticky flag since the last call); raises on EHIP."""
    rc = _lib.saef_status(layout.handle, _stream(stream))
    if rc not in (OK, ERANGE):
        raise SaefError("saef_status", rc)
    return rc


def saef_profile_enable(layout: Layout, capacity: int, kinds=PROFILE_KINDS,
                        every: int = 1) -> None:
    """Time the kernels of the given kinds (names from PROFILE_KINDS) in the
    next saef_round calls, up to `capacity` launches; every > 1 times only
    every `every`-th dispatch of each kind."""
    mask = 0
    for k in kinds:
        mask |= 1 << PROFILE_KINDS.index(k)
    _check("saef_profile_enable",
           _lib.saef_profile_enable(layout.handle, int(capacity), mask, int(every)))


def saef_profile_read(layout: Layout) -> dict:
    """{kind: (launches timed, summed milliseconds)} since the last read."""
    counts = (ctypes.c_int32 * len(PROFILE_KINDS))()
    ms = (ctypes.c_double * len(PROFILE_KINDS))()
    _check("saef_profile_read", _lib.saef_profile_read(layout.handle, counts, ms))
    return {k: (counts[i], ms[i]) for i, k in enumerate(PROFILE_KINDS)}


def saef_stream_probe(a, b, c, stream=None) -> None:
    """c = a + b over equal-size contiguous fp32 device tensors (the HBM
    ceiling of the compression's streaming pattern; measurement aid); with
    b None, c = a (c may be a itself: one read and one write in place)."""
    n = a.numel()
    if (b is not None and b.numel() != n) or c.numel() != n:
        raise ValueError("saef_stream_probe: a, b and c must have the same size")
    _check("saef_stream_probe", _lib.saef_stream_probe(_f(a), None if b is None else _f(b),
                                                       _f(c), n, _stream(stream)))


def raw_library() -> ctypes.CDLL:
    """The loaded ctypes library (for callers that pass raw pointers)."""
    return _lib
