"""The C oracle run piecewise on a pool of threads, for the full-size parity
tests (test infrastructure only).

Every step of an iteration of Algorithm 1 with layer-wise compression acts on
one tensor alone -- the scales are per tensor, everything else is elementwise
-- and the worker compression acts on one worker alone.  So the oracle's own
functions, called on single-tensor layouts that address the same full
buffers, give the result of one call over the whole layout:

- first half (error averaging when due, step ahead): oracle_round_begin on
  element chunks (a tensor or a 64-aligned piece of one), all K workers;
- worker compression: oracle_compress per (tensor, worker) with K = 1 on the
  worker's rows;
- server: oracle_aggregate per tensor over the K messages.

The calls touch disjoint elements, words and scales, and ctypes releases the
GIL during a foreign call, so they run in parallel threads.  The equivalence
with oracle_round on the whole layout is checked bit for bit by a CPU test.
Nothing here does any of the method's arithmetic.
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from oracle import oracle as O
from paper_2008_05823_amd import workloads as W

_i64p = ctypes.POINTER(ctypes.c_int64)


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


class SplitOracle:
    """Host state of Algorithm 1 (SAEF branch, mu = 0) advanced by the C
    oracle in pieces.  Arrays as in tests.gpu_harness.OracleState."""

    def __init__(self, w: W.Workload, x0: np.ndarray | None = None, threads: int | None = None,
                 chunk: int = 1 << 22):
        self.w = w
        self.K = w.K
        off, n, d_pad = w.layout()
        self.off, self.n, self.d_pad = off, n, d_pad
        self.L = w.L
        self.lib = O.lib()
        self.threads = threads or default_threads()
        K, L = self.K, self.L
        self.x = (W.initial_x(w) if x0 is None else x0).copy()
        self.e = np.zeros((K, d_pad), np.float32)
        self.e_srv = np.zeros(d_pad, np.float32)
        self.xh = np.zeros((K, d_pad), np.float32)
        self.signs = np.zeros((K, d_pad // 64), np.uint64)
        self.srv_signs = np.zeros(d_pad // 64, np.uint64)
        # per-tensor scale columns (contiguous, the oracle's (K, 1) layout)
        self._sc = [np.zeros(K, np.float32) for _ in range(L)]
        self._ssc = np.zeros(L, np.float32)
        # single-tensor layouts, largest tensors first (load balance)
        self._lay = [(np.array([off[l]], np.int64), np.array([n[l]], np.int64)) for l in range(L)]
        self._order = sorted(range(L), key=lambda l: -int(n[l]))
        # element chunks of the first half: pieces of at most `chunk` elements
        chunk = max(64, chunk // 64 * 64)
        self._chunks = []
        for l in self._order:
            for a in range(0, int(n[l]), chunk):
                self._chunks.append((np.array([off[l] + a], np.int64),
                                     np.array([min(chunk, int(n[l]) - a)], np.int64)))

    @property
    def scales(self) -> np.ndarray:
        return np.stack(self._sc, axis=1)  # (K, L)

    @property
    def srv_scales(self) -> np.ndarray:
        return self._ssc.copy()

    @staticmethod
    def _p(a: np.ndarray, elem_off: int = 0) -> int:
        assert a.flags["C_CONTIGUOUS"]
        return a.ctypes.data + elem_off * a.itemsize

    def _run(self, fn, items):
        with ThreadPoolExecutor(self.threads) as ex:
            rcs = list(ex.map(fn, items))
        bad = [rc for rc in rcs if rc != O.OK]
        assert not bad, bad[:4]

    def round(self, t: int, g: np.ndarray, period: int | None = None, mode: int | None = None):
        w, lib, K = self.w, self.lib, self.K
        period = w.period if period is None else period
        mode = w.mode if mode is None else mode
        assert g.shape == (K, self.d_pad) and g.dtype == np.float32 and g.flags["C_CONTIGUOUS"]
        d_pad, Wd = self.d_pad, self.d_pad // 64
        lr = ctypes.c_float(np.float32(w.lr))

        def begin(ch):
            o, n = ch
            return lib.oracle_round_begin(1, o.ctypes.data, n.ctypes.data, d_pad, t, period, K,
                                          mode, 1, self._p(self.e), self._p(self.e_srv),
                                          self._p(self.x), self._p(self.xh), None)

        self._run(begin, self._chunks)

        def compress(item):
            l, k = item
            o, n = self._lay[l]
            return lib.oracle_compress(1, o.ctypes.data, n.ctypes.data, d_pad, 1, lr,
                                       self._p(g, k * d_pad), self._p(self.e, k * d_pad),
                                       self._p(self.signs, k * Wd), self._p(self._sc[l], k))

        self._run(compress, [(l, k) for l in self._order for k in range(K)])

        def aggregate(l):
            o, n = self._lay[l]
            return lib.oracle_aggregate(1, o.ctypes.data, n.ctypes.data, d_pad, K, mode,
                                        self._p(self.signs), self._p(self._sc[l]), None,
                                        self._p(self.e_srv) if mode == 1 else None,
                                        self._p(self.srv_signs) if mode == 1 else None,
                                        self._p(self._ssc, l) if mode == 1 else None,
                                        self._p(self.x))

        self._run(aggregate, self._order)


def rows_equal(a: np.ndarray, b: np.ndarray, threads: int | None = None) -> bool:
    """Bit equality of two same-shape arrays, compared in row blocks on a
    thread pool (numpy releases the GIL for the comparisons)."""
    assert a.shape == b.shape and a.dtype.itemsize == b.dtype.itemsize
    ua = a.reshape(-1).view(np.uint8 if a.dtype.itemsize == 1 else f"u{a.dtype.itemsize}")
    ub = b.reshape(-1).view(ua.dtype)
    n = ua.size
    step = max(1 << 20, -(-n // (4 * (threads or default_threads()))))
    with ThreadPoolExecutor(threads or default_threads()) as ex:
        res = list(ex.map(lambda s: bool(np.array_equal(ua[s:s + step], ub[s:s + step])),
                          range(0, n, step)))
    return all(res)
