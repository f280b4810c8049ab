"""Helpers of the GPU parity tests: device buffers for a workload, the same
iteration run by the HIP library and by the CPU oracle, and comparisons.

The oracle and the HIP path share nothing but the inputs drawn by
paper_2008_05823_amd.workloads; expected values always come from the oracle.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O
from paper_2008_05823_amd import workloads as W

REL_TOL, ABS_TOL = 1e-6, 1e-7   # acceptance bound for fp32 state


def dev(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint64:
        a = a.view(np.int64)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t: torch.Tensor, like=np.float32) -> np.ndarray:
    a = t.detach().cpu().numpy()
    if like == np.uint64:
        a = a.view(np.uint64)
    return a


def tensor_word_mask(off, n, d_pad) -> np.ndarray:
    m = np.zeros(d_pad // 64, bool)
    for o, nl in zip(off, n):
        m[o // 64:o // 64 + (nl + 63) // 64] = True
    return m


def assert_f32_equal(got: np.ndarray, want: np.ndarray, mask: np.ndarray, what: str):
    """Bit-exact equality on the masked elements (the design gives identical
    IEEE operations on both sides); the report also shows the spec tolerance."""
    g = got[..., mask]
    w = want[..., mask]
    same = g.view(np.uint32) == w.view(np.uint32)
    if same.all():
        return
    tol_ok = np.abs(g.astype(np.float64) - w) <= ABS_TOL + REL_TOL * np.abs(w.astype(np.float64))
    bad = np.argwhere(~same)
    first = tuple(bad[0])
    raise AssertionError(
        f"{what}: {int((~same).sum())} of {same.size} values differ from the oracle "
        f"({int((~tol_ok).sum())} beyond 1e-6 rel/1e-7 abs); first at {first}: "
        f"got {g[first]!r} want {w[first]!r}")


def assert_words_equal(got: np.ndarray, want: np.ndarray, wmask: np.ndarray, what: str):
    g = got[..., wmask]
    w = want[..., wmask]
    if not np.array_equal(g, w):
        bad = np.argwhere(g != w)
        first = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} sign words differ; first at {first}: "
                             f"got {int(g[first]):#x} want {int(w[first]):#x}")


class OracleState:
    """Host state of Algorithm 1 advanced by the C oracle (with momentum
    constant mu when given)."""

    def __init__(self, w: W.Workload, x0: np.ndarray | None = None, K: int | None = None,
                 mu: float | None = None):
        self.w = w
        self.mu = mu
        self.K = w.K if K is None else K
        off, n, d_pad = w.layout()
        self.orc = O.Oracle(off, n, d_pad)
        self.x = (W.initial_x(w) if x0 is None else x0).copy()
        self.e = np.zeros((self.K, d_pad), np.float32)
        self.e_srv = np.zeros(d_pad, np.float32)
        self.xh = np.zeros((self.K, d_pad), np.float32)
        self.signs = np.zeros((self.K, d_pad // 64), np.uint64)
        self.scales = np.zeros((self.K, w.L), np.float32)
        self.srv_signs = np.zeros(d_pad // 64, np.uint64)
        self.srv_scales = np.zeros(w.L, np.float32)
        self.m = np.zeros((self.K, d_pad), np.float32) if mu is not None else None

    def round(self, t: int, g: np.ndarray, period=None, mode=None):
        w = self.w
        period = w.period if period is None else period
        mode = w.mode if mode is None else mode
        if self.mu is None:
            rc = self.orc.round(t, period, self.K, np.float32(w.lr), mode, g, self.e, self.e_srv,
                                self.x, self.xh, self.signs, self.scales, self.srv_signs,
                                self.srv_scales)
        else:
            rc = self.orc.round_momentum(t, period, self.K, np.float32(w.lr),
                                         np.float32(self.mu), mode, g, self.m, self.e,
                                         self.e_srv, self.x, self.xh, self.signs, self.scales,
                                         self.srv_signs, self.srv_scales)
        assert rc == O.OK, rc

    def begin(self, t: int, variant: int, period=None, mode=None, mismatch=True):
        """First half of iteration t; returns the 2 L mismatch bounds (or None)."""
        w = self.w
        period = w.period if period is None else period
        mode = w.mode if mode is None else mode
        mism = np.full(2 * w.L, np.nan) if mismatch else None
        rc = self.orc.round_begin(t, period, self.K, mode, variant, self.e, self.e_srv, self.x,
                                  self.xh, mism)
        assert rc == O.OK, rc
        return mism

    def end(self, t: int, g: np.ndarray, mode=None):
        w = self.w
        mode = w.mode if mode is None else mode
        mu = 0.0 if self.mu is None else np.float32(self.mu)
        rc = self.orc.round_end(self.K, np.float32(w.lr), mu, mode, g, self.m, self.e,
                                self.e_srv, self.x, self.signs, self.scales, self.srv_signs,
                                self.srv_scales)
        assert rc == O.OK, rc


class GpuState:
    """Device buffers of one workload driven through the HIP library (with
    momentum constant mu when given)."""

    def __init__(self, w: W.Workload, x0: np.ndarray | None = None, K: int | None = None,
                 k_max: int | None = None, mu: float | None = None):
        from paper_2008_05823_amd import saef
        self.saef = saef
        self.w = w
        self.mu = mu
        self.K = w.K if K is None else K
        off, n, d_pad = w.layout()
        self.off, self.n, self.d_pad = off, n, d_pad
        self.layout = saef.Layout(off, n, d_pad, k_max or self.K)
        f32 = dict(dtype=torch.float32, device="cuda")
        i64 = dict(dtype=torch.int64, device="cuda")
        self.x = dev(W.initial_x(w) if x0 is None else x0)
        self.e = torch.zeros((self.K, d_pad), **f32)
        self.e_srv = torch.zeros(d_pad, **f32)
        self.xh = torch.zeros((self.K, d_pad), **f32)
        self.signs = torch.zeros((self.K, d_pad // 64), **i64)
        self.scales = torch.zeros((self.K, w.L), **f32)
        self.srv_signs = torch.zeros(d_pad // 64, **i64)
        self.srv_scales = torch.zeros(w.L, **f32)
        self.g = torch.zeros((self.K, d_pad), **f32)
        self.m = torch.zeros((self.K, d_pad), **f32) if mu is not None else None

    def round(self, t: int, g: np.ndarray | torch.Tensor, period=None, mode=None):
        w = self.w
        if isinstance(g, np.ndarray):
            self.g.copy_(torch.from_numpy(g))
        else:
            self.g.copy_(g)
        period = w.period if period is None else period
        mode = w.mode if mode is None else mode
        if self.mu is None:
            self.saef.saef_round(self.layout, t, period, self.K, w.lr, mode, self.g, self.e,
                                 self.e_srv, self.x, self.xh, self.signs, self.scales,
                                 self.srv_signs, self.srv_scales)
        else:
            self.saef.saef_round_momentum(self.layout, t, period, self.K, w.lr, self.mu, mode,
                                          self.g, self.m, self.e, self.e_srv, self.x, self.xh,
                                          self.signs, self.scales, self.srv_signs,
                                          self.srv_scales)

    def begin(self, t: int, variant: int, period=None, mode=None, mismatch=True):
        """First half of iteration t (EF writes row 0 of xh); returns the 2 L
        mismatch bounds downloaded to the host (or None)."""
        w = self.w
        period = w.period if period is None else period
        mode = w.mode if mode is None else mode
        mism = torch.full((2 * w.L,), float("nan"), dtype=torch.float64,
                          device="cuda") if mismatch else None
        xh = self.xh if variant == self.saef.VARIANT_SAEF else self.xh[0]
        self.saef.saef_round_begin(self.layout, t, period, self.K, mode, variant, self.e,
                                   self.e_srv, self.x, xh, self.signs, self.scales,
                                   self.srv_signs, self.srv_scales, mism)
        return None if mism is None else mism.cpu().numpy()

    def end(self, t: int, g, period=None, mode=None):
        w = self.w
        if isinstance(g, np.ndarray):
            self.g.copy_(torch.from_numpy(g))
        else:
            self.g.copy_(g)
        period = w.period if period is None else period
        mode = w.mode if mode is None else mode
        self.saef.saef_round_end(self.layout, t, period, self.K, w.lr,
                                 0.0 if self.mu is None else self.mu, mode, self.g, self.m,
                                 self.e, self.e_srv, self.x, self.signs, self.scales,
                                 self.srv_signs, self.srv_scales)

    def plain(self, mode=None) -> dict:
        """Materialized (plain) state, downloaded to the host."""
        mode = self.w.mode if mode is None else mode
        e_out = torch.zeros_like(self.e)
        es_out = torch.zeros_like(self.e_srv)
        x_out = torch.zeros_like(self.x)
        self.saef.saef_materialize(self.layout, self.K, mode, self.e, self.e_srv, self.x,
                                   self.signs, self.scales, self.srv_signs, self.srv_scales,
                                   e_out, es_out, x_out)
        torch.cuda.synchronize()
        out = dict(e=host(e_out), e_srv=host(es_out), x=host(x_out), xh=host(self.xh),
                   signs=host(self.signs, np.uint64), scales=host(self.scales),
                   srv_signs=host(self.srv_signs, np.uint64), srv_scales=host(self.srv_scales))
        if self.m is not None:
            out["m"] = host(self.m)
        return out

    def status(self) -> int:
        return self.saef.saef_status(self.layout)


def compare_state(gpu: dict, orc: OracleState, t: int, what: str = ""):
    w = orc.w
    off, n, d_pad = w.layout()
    m = W.tensor_mask(w)
    wm = tensor_word_mask(off, n, d_pad)
    tag = f"{what} t={t}"
    assert_words_equal(gpu["signs"], orc.signs, wm, f"{tag} worker sign words")
    assert_f32_equal(gpu["scales"], orc.scales, np.ones(w.L, bool), f"{tag} worker scales")
    assert_f32_equal(gpu["e"], orc.e, m, f"{tag} worker errors")
    assert_f32_equal(gpu["xh"], orc.xh, m, f"{tag} step-ahead weights")
    assert_f32_equal(gpu["x"], orc.x, m, f"{tag} weights")
    if orc.m is not None:
        assert_f32_equal(gpu["m"], orc.m, m, f"{tag} momentum buffers")
    if w.mode == 1:
        assert_words_equal(gpu["srv_signs"], orc.srv_signs, wm, f"{tag} server sign words")
        assert_f32_equal(gpu["srv_scales"], orc.srv_scales, np.ones(w.L, bool),
                         f"{tag} server scales")
        assert_f32_equal(gpu["e_srv"], orc.e_srv, m, f"{tag} server error")


def mismatch_tol(w: W.Workload, K: int) -> np.ndarray:
    """Per-entry bound on |gpu - oracle| / value for the 2 L mismatch sums:
    every term is the same binary64 value on both sides and non-negative, so
    two summation orders of N terms differ by at most 2 (N - 1) 2^-53 of the
    sum (N = n_l for the EF bound, n_l K for the step-ahead bound)."""
    n = w.sizes.astype(np.float64)
    return np.concatenate([2 * n, 2 * n * K]) * 2.0 ** -53 + 4 * 2.0 ** -53


def assert_mismatch_close(got: np.ndarray, want: np.ndarray, w: W.Workload, K: int, what: str):
    rel = mismatch_tol(w, K)
    err = np.abs(got - want)
    ok = err <= rel * np.abs(want) + 1e-300
    if not ok.all():
        i = int(np.argwhere(~ok)[0][0])
        raise AssertionError(f"{what}: mismatch bound {i} got {got[i]!r} want {want[i]!r} "
                             f"(rel err {err[i] / max(abs(want[i]), 1e-300):.3g}, "
                             f"bound {rel[i]:.3g})")
