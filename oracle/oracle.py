"""ctypes wrapper around the C oracle -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg
may import this module.  The product library (``paper_2008_05823_amd``) never
does, and this module never imports the product library.

All arrays are host numpy arrays: float32 value buffers of shape (K, d_pad) or
(d_pad,), uint64 sign words of shape (K, d_pad // 64) or (d_pad // 64,), float32
scales of shape (K, L) or (L,).  Every call works in place on the arrays passed,
like the C functions it wraps, and returns the C status code (0 ok, -1 invalid
arguments, -2 value out of the exact-sum range).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "saef_oracle.c")
LIB = os.path.join(HERE, "liboracle_saef.so")

OK, EINVAL, ERANGE = 0, -1, -2

GCC_FLAGS = ["-O1", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
             "-fno-fast-math", "-Wall", "-Wextra", "-Werror"]


def build(src: str = SRC, out: str = LIB, werror: bool = True) -> str:
    """Compile the oracle with gcc (plain C, IEEE arithmetic, no contraction)."""
    flags = [f for f in GCC_FLAGS if werror or f != "-Werror"]
    cmd = ["gcc", *flags, "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_P = ctypes.c_void_p
_I64P = ctypes.POINTER(ctypes.c_int64)


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    lay = [i32, _P, _P, i64]
    sigs = {
        "oracle_l1_fixed": [_P, i64, _P, _P],
        "oracle_compress": lay + [i32, f32, _P, _P, _P, _P],
        "oracle_aggregate": lay + [i32, i32, _P, _P, _P, _P, _P, _P, _P],
        "oracle_step_ahead": lay + [i32, _P, _P, _P],
        "oracle_error_average": lay + [i32, _P],
        "oracle_round": lay + [i64, i64, i32, f32, i32, _P, _P, _P, _P, _P, _P, _P, _P, _P],
        "oracle_compress_momentum": lay + [i32, f32, f32, _P, _P, _P, _P, _P],
        "oracle_round_momentum": lay + [i64, i64, i32, f32, f32, i32, _P, _P, _P, _P, _P, _P,
                                        _P, _P, _P, _P],
        "oracle_mismatch": lay + [i32, _P, _P, _P, _P],
        "oracle_round_begin": lay + [i64, i64, i32, i32, i32, _P, _P, _P, _P, _P],
        "oracle_round_end": lay + [i32, f32, f32, i32, _P, _P, _P, _P, _P, _P, _P, _P, _P],
        "oracle_topk_compress": lay + [i32, f32, f32, _P, _P, _P, _P, _P, _P, _P],
        "oracle_topk_aggregate": lay + [i32, i32, _P, _P, _P, _P, _P, _P, _P, _P, _P],
        "oracle_topk_round": lay + [i64, i64, i32, f32, f32, i32, _P, _P, _P, _P, _P, _P, _P, _P,
                                    _P, _P, _P, _P, _P],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.oracle_scale_from_sum.argtypes = [ctypes.c_uint64, ctypes.c_uint64, i64]
    lib.oracle_scale_from_sum.restype = ctypes.c_float
    return lib


_lib = None


def lib(path: str = LIB) -> ctypes.CDLL:
    """Load the built oracle (building it first if no library exists yet)."""
    global _lib
    if _lib is None or path != LIB:
        if not os.path.exists(path):
            build(out=path)
        handle = _bind(ctypes.CDLL(path))
        if path != LIB:
            return handle
        _lib = handle
    return _lib


def _ptr(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle buffers must be contiguous"
    return a.ctypes.data


class Oracle:
    """The oracle bound to one tensor layout (offsets, sizes, d_pad)."""

    def __init__(self, offsets, sizes, d_pad: int, libpath: str = LIB):
        self.off = np.ascontiguousarray(offsets, dtype=np.int64)
        self.n = np.ascontiguousarray(sizes, dtype=np.int64)
        self.L = int(self.off.size)
        self.d_pad = int(d_pad)
        self.lib = lib(libpath)

    def _lay(self):
        return (self.L, _ptr(self.off), _ptr(self.n), self.d_pad)

    def compress(self, K, lr, g, e, signs, scales):
        _check(g, np.float32), _check(e, np.float32)
        _check(signs, np.uint64), _check(scales, np.float32)
        return self.lib.oracle_compress(*self._lay(), K, lr, _ptr(g), _ptr(e),
                                        _ptr(signs), _ptr(scales))

    def aggregate(self, K, mode, signs, scales, x, e_srv=None, srv_signs=None,
                  srv_scales=None, avg=None):
        return self.lib.oracle_aggregate(*self._lay(), K, mode, _ptr(signs), _ptr(scales),
                                         _ptr(avg), _ptr(e_srv), _ptr(srv_signs),
                                         _ptr(srv_scales), _ptr(x))

    def compress_momentum(self, K, lr, mu, g, m, e, signs, scales):
        return self.lib.oracle_compress_momentum(*self._lay(), K, lr, mu, _ptr(g), _ptr(m),
                                                 _ptr(e), _ptr(signs), _ptr(scales))

    def round_momentum(self, t, period, K, lr, mu, mode, g, m, e, e_srv, x, xh, signs, scales,
                       srv_signs, srv_scales):
        return self.lib.oracle_round_momentum(*self._lay(), t, period, K, lr, mu, mode, _ptr(g),
                                              _ptr(m), _ptr(e), _ptr(e_srv), _ptr(x), _ptr(xh),
                                              _ptr(signs), _ptr(scales), _ptr(srv_signs),
                                              _ptr(srv_scales))

    def mismatch(self, K, e, e_srv=None):
        """(ef, saef): per-tensor gradient-mismatch bounds (binary64)."""
        ef = np.zeros(self.L, np.float64)
        saef = np.zeros(self.L, np.float64)
        rc = self.lib.oracle_mismatch(*self._lay(), K, _ptr(e), _ptr(e_srv), _ptr(ef),
                                      _ptr(saef))
        assert rc == 0, rc
        return ef, saef

    def round_begin(self, t, period, K, mode, variant, e, e_srv, x, xh, mismatch=None):
        return self.lib.oracle_round_begin(*self._lay(), t, period, K, mode, variant, _ptr(e),
                                           _ptr(e_srv), _ptr(x), _ptr(xh), _ptr(mismatch))

    def round_end(self, K, lr, mu, mode, g, m, e, e_srv, x, signs, scales, srv_signs,
                  srv_scales):
        return self.lib.oracle_round_end(*self._lay(), K, lr, mu, mode, _ptr(g), _ptr(m),
                                         _ptr(e), _ptr(e_srv), _ptr(x), _ptr(signs),
                                         _ptr(scales), _ptr(srv_signs), _ptr(srv_scales))

    def topk_compress(self, K, lr, mu, keep, g, m, e, sel, rank, vals):
        keep = np.ascontiguousarray(keep, dtype=np.int64)
        return self.lib.oracle_topk_compress(*self._lay(), K, lr, mu, _ptr(keep), _ptr(g),
                                             _ptr(m), _ptr(e), _ptr(sel), _ptr(rank),
                                             _ptr(vals))

    def topk_aggregate(self, K, mode, keep, sel, vals, x, e_srv=None, srv_sel=None,
                       srv_rank=None, srv_vals=None, avg=None):
        keep = np.ascontiguousarray(keep, dtype=np.int64)
        return self.lib.oracle_topk_aggregate(*self._lay(), K, mode, _ptr(keep), _ptr(sel),
                                              _ptr(vals), _ptr(avg), _ptr(e_srv), _ptr(srv_sel),
                                              _ptr(srv_rank), _ptr(srv_vals), _ptr(x))

    def topk_round(self, t, period, K, lr, mu, mode, keep, g, m, e, e_srv, x, xh, sel, rank,
                   vals, srv_sel, srv_rank, srv_vals):
        keep = np.ascontiguousarray(keep, dtype=np.int64)
        return self.lib.oracle_topk_round(*self._lay(), t, period, K, lr, mu, mode, _ptr(keep),
                                          _ptr(g), _ptr(m), _ptr(e), _ptr(e_srv), _ptr(x),
                                          _ptr(xh), _ptr(sel), _ptr(rank), _ptr(vals),
                                          _ptr(srv_sel), _ptr(srv_rank), _ptr(srv_vals))

    def step_ahead(self, K, x, e, xh):
        return self.lib.oracle_step_ahead(*self._lay(), K, _ptr(x), _ptr(e), _ptr(xh))

    def error_average(self, K, e):
        return self.lib.oracle_error_average(*self._lay(), K, _ptr(e))

    def round(self, t, period, K, lr, mode, g, e, e_srv, x, xh, signs, scales,
              srv_signs, srv_scales):
        return self.lib.oracle_round(*self._lay(), t, period, K, lr, mode, _ptr(g), _ptr(e),
                                     _ptr(e_srv), _ptr(x), _ptr(xh), _ptr(signs),
                                     _ptr(scales), _ptr(srv_signs), _ptr(srv_scales))


def l1_fixed(v) -> tuple[int, int]:
    """(status, S) with S = sum floor(|v_i| 2^80) as a Python int."""
    v = np.ascontiguousarray(v, dtype=np.float32)
    hi, lo = ctypes.c_uint64(), ctypes.c_uint64()
    rc = lib().oracle_l1_fixed(_ptr(v), v.size, ctypes.byref(hi), ctypes.byref(lo))
    return rc, (hi.value << 64) | lo.value


def scale_from_sum(S: int, n: int) -> np.float32:
    return np.float32(lib().oracle_scale_from_sum(S >> 64, S & (2**64 - 1), n))


def _check(a, dtype):
    if a is not None and a.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {a.dtype}")
