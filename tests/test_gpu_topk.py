"""Parity of the layer-wise Top-K path of the HIP library with the CPU oracle
(needs an MI355X).

The kept set is a discrete decision taken on exact keys on both sides, so
everything is compared bit for bit: selection words, rank words, kept
values, errors, weights.  Inputs include heavy ties (few distinct
magnitudes), exact zeros of both signs, tensors spanning many tile groups
(and super-groups above 4096 tiles), ragged sizes, and a data scale that
jumps across the histogram window between calls.
"""
import zlib

import numpy as np
import pytest
import torch

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H

pytestmark = pytest.mark.gpu

LR = np.float32(0.1)
ADVERSARIAL = [1, 3, 4, 10, 63, 64, 65, 255, 256, 257, 4095, 4096, 4097, 8193, 12345]


def _case(msg):
    print(f"[case] {msg}", flush=True)


def _tie_values(rng, shape, levels=4):
    """Values with few distinct magnitudes (long runs of equal keys), signed
    zeros included."""
    mag = rng.integers(0, levels, shape).astype(np.float32) * np.float32(0.25)
    sign = np.where(rng.random(shape) < 0.5, -1.0, 1.0).astype(np.float32)
    return (mag * sign).astype(np.float32)


class TopkOracle:
    def __init__(self, w, keep, K=None, x0=None, mu=None):
        from oracle import oracle as O
        self.O = O
        self.w, self.K = w, (w.K if K is None else K)
        off, n, d_pad = w.layout()
        self.orc = O.Oracle(off, n, d_pad)
        self.keep = np.asarray(keep, np.int64)
        total = int(self.keep.sum())
        Wd = d_pad // 64
        self.x = (W.initial_x(w) if x0 is None else x0).copy()
        self.e = np.zeros((self.K, d_pad), np.float32)
        self.m = np.zeros((self.K, d_pad), np.float32) if mu is not None else None
        self.mu = mu
        self.e_srv = np.zeros(d_pad, np.float32)
        self.xh = np.zeros((self.K, d_pad), np.float32)
        self.sel = np.zeros((self.K, Wd), np.uint64)
        self.rank = np.zeros((self.K, Wd), np.uint32)
        self.vals = np.zeros((self.K, total), np.float32)
        self.srv_sel = np.zeros(Wd, np.uint64)
        self.srv_rank = np.zeros(Wd, np.uint32)
        self.srv_vals = np.zeros(total, np.float32)

    def round(self, t, g, period=None, mode=None):
        w = self.w
        mu = np.float32(0.0 if self.mu is None else self.mu)
        rc = self.orc.topk_round(t, w.period if period is None else period, self.K,
                                 np.float32(w.lr), mu, w.mode if mode is None else mode,
                                 self.keep, g, self.m, self.e, self.e_srv, self.x, self.xh,
                                 self.sel, self.rank, self.vals, self.srv_sel, self.srv_rank,
                                 self.srv_vals)
        assert rc == self.O.OK, rc

    def begin(self, t, variant, mismatch=True):
        w = self.w
        mism = np.full(2 * w.L, np.nan) if mismatch else None
        rc = self.orc.round_begin(t, w.period, self.K, w.mode, variant, self.e, self.e_srv, self.x,
                                  self.xh, mism)
        assert rc == self.O.OK, rc
        return mism

    def end(self, g):
        w = self.w
        mu = np.float32(0.0 if self.mu is None else self.mu)
        rc = self.orc.topk_compress(self.K, np.float32(w.lr), mu, self.keep, g, self.m, self.e,
                                    self.sel, self.rank, self.vals)
        assert rc == self.O.OK, rc
        rc = self.orc.topk_aggregate(self.K, w.mode, self.keep, self.sel, self.vals, self.x,
                                     self.e_srv, self.srv_sel, self.srv_rank, self.srv_vals)
        assert rc == self.O.OK, rc


class TopkGpu:
    def __init__(self, w, keep, K=None, x0=None, mu=None):
        from paper_2008_05823_amd import saef
        self.saef = saef
        self.w, self.K, self.mu = w, (w.K if K is None else K), mu
        off, n, d_pad = w.layout()
        self.layout = saef.Layout(off, n, d_pad, self.K)
        self.plan = saef.TopK(self.layout, keep)
        total = self.plan.total
        f32 = dict(dtype=torch.float32, device="cuda")
        Wd = d_pad // 64
        self.x = H.dev(W.initial_x(w) if x0 is None else x0)
        self.e = torch.zeros((self.K, d_pad), **f32)
        self.m = torch.zeros((self.K, d_pad), **f32) if mu is not None else None
        self.e_srv = torch.zeros(d_pad, **f32)
        self.xh = torch.zeros((self.K, d_pad), **f32)
        self.g = torch.zeros((self.K, d_pad), **f32)
        self.sel = torch.zeros((self.K, Wd), dtype=torch.int64, device="cuda")
        self.rank = torch.zeros((self.K, Wd), dtype=torch.int32, device="cuda")
        self.vals = torch.zeros((self.K, total), **f32)
        self.srv_sel = torch.zeros(Wd, dtype=torch.int64, device="cuda")
        self.srv_rank = torch.zeros(Wd, dtype=torch.int32, device="cuda")
        self.srv_vals = torch.zeros(total, **f32)

    def round(self, t, g, period=None, mode=None):
        w = self.w
        self.g.copy_(torch.from_numpy(g) if isinstance(g, np.ndarray) else g)
        self.saef.saef_topk_round(self.plan, t, w.period if period is None else period, self.K,
                                  w.lr, 0.0 if self.mu is None else self.mu,
                                  w.mode if mode is None else mode, self.g, self.m, self.e,
                                  self.e_srv, self.x, self.xh, self.sel, self.rank, self.vals,
                                  self.srv_sel, self.srv_rank, self.srv_vals)

    def begin(self, t, variant, mismatch=True):
        w = self.w
        mism = torch.full((2 * w.L,), float("nan"), dtype=torch.float64,
                          device="cuda") if mismatch else None
        xh = self.xh if variant == self.saef.VARIANT_SAEF else self.xh[0]
        self.saef.saef_topk_round_begin(self.plan, t, w.period, self.K, w.mode, variant, self.e,
                                        self.sel, self.e_srv, self.x, xh, mism)
        return None if mism is None else mism.cpu().numpy()

    def end(self, t, g):
        w = self.w
        self.g.copy_(torch.from_numpy(g) if isinstance(g, np.ndarray) else g)
        self.saef.saef_topk_round_end(self.plan, t, w.period, self.K, w.lr,
                                      0.0 if self.mu is None else self.mu, w.mode, self.g, self.m,
                                      self.e, self.e_srv, self.x, self.sel, self.rank, self.vals,
                                      self.srv_sel, self.srv_rank, self.srv_vals)

    def plain_e(self):
        """The plain worker errors (a materialized copy; the state itself
        stays pending)."""
        e = self.e.clone()
        self.saef.saef_topk_materialize(self.plan, self.K, e, self.sel)
        return e

    def status(self):
        return self.saef.saef_status(self.layout)


def _u32(t):
    return t.cpu().numpy().view(np.uint32)


def compare_topk(gpu: TopkGpu, orc: TopkOracle, t, what, mode=1):
    w = orc.w
    off, n, d_pad = w.layout()
    m = W.tensor_mask(w)
    wm = H.tensor_word_mask(off, n, d_pad)
    tag = f"{what} t={t}"
    torch.cuda.synchronize()
    H.assert_words_equal(H.host(gpu.sel, np.uint64), orc.sel, wm, f"{tag} worker selection")
    got_rank = _u32(gpu.rank)
    assert np.array_equal(got_rank[:, wm], orc.rank[:, wm]), f"{tag} worker rank words"
    H.assert_f32_equal(H.host(gpu.vals), orc.vals, np.ones(orc.vals.shape[-1], bool),
                       f"{tag} worker values")
    H.assert_f32_equal(H.host(gpu.plain_e()), orc.e, m, f"{tag} worker errors")
    H.assert_f32_equal(H.host(gpu.xh), orc.xh, m, f"{tag} step-ahead weights")
    H.assert_f32_equal(H.host(gpu.x), orc.x, m, f"{tag} weights")
    if orc.m is not None:
        H.assert_f32_equal(H.host(gpu.m), orc.m, m, f"{tag} momentum buffers")
    if mode == 1:
        H.assert_words_equal(H.host(gpu.srv_sel, np.uint64), orc.srv_sel, wm,
                             f"{tag} server selection")
        assert np.array_equal(_u32(gpu.srv_rank)[wm], orc.srv_rank[wm]), f"{tag} server ranks"
        H.assert_f32_equal(H.host(gpu.srv_vals), orc.srv_vals,
                           np.ones(orc.srv_vals.shape[-1], bool), f"{tag} server values")
        H.assert_f32_equal(H.host(gpu.e_srv), orc.e_srv, m, f"{tag} server error")


COMPRESS_CASES = {
    # name: (K, sizes, keep rule, value source)
    "adversarial_1pct": (3, ADVERSARIAL, 1, "grad"),
    "adversarial_keep_all": (2, ADVERSARIAL, 100, "grad"),
    "ties_10pct": (4, [300_000, 77, 64, 4097], 10, "ties"),
    "ties_keep_one": (2, [5000, 1, 130], "one", "ties"),
    "many_chunks": (2, [64 * 65536 + 4097, 33], 5, "grad"),   # 2050 tiles: 33 tile groups
    "big_ties": (2, [70 * 65536 + 5], 1, "ties"),              # tie cut in a later group
    "super_groups": (1, [4097 * 2048 + 77, 100], 1, "grad"),   # > 4096 tiles: super-groups
}


def _keep(w, rule):
    if rule == "one":
        return np.ones(w.L, np.int64)
    return W.topk_keep(w, rule)


COMPRESS_RUNS = [(name, False) for name in COMPRESS_CASES] + [
    ("adversarial_1pct", True), ("ties_10pct", True)]


@pytest.mark.parametrize("name,momentum", COMPRESS_RUNS,
                         ids=[f"{n}-{'momentum' if m else 'plain'}" for n, m in COMPRESS_RUNS])
def test_topk_compress_parity(name, momentum):
    K, sizes, rule, src = COMPRESS_CASES[name]
    _case(f"topk compress {name} K={K} momentum={momentum}")
    seed = zlib.crc32(name.encode())
    w = W.custom(sizes, K=K, scale_range=(1e-3, 1.0), seed=seed % 1000 + 11)
    keep = _keep(w, rule)
    off, n, d_pad = w.layout()
    msk = W.tensor_mask(w)
    rng = np.random.default_rng(seed)
    if src == "ties":
        g = _tie_values(rng, (K, d_pad))
        e = _tie_values(rng, (K, d_pad))
    else:
        g = W.gradients(w, 0)
        e = (rng.standard_normal((K, d_pad)) * 0.01).astype(np.float32)
    g[:, ~msk] = np.nan
    e[:, ~msk] = np.nan   # padding must stay untouched
    mu = 0.9 if momentum else None
    m0 = _tie_values(rng, (K, d_pad)) if momentum else None
    orc = TopkOracle(w, keep, mu=mu)
    orc.e[:] = e
    if momentum:
        orc.m[:] = m0
    rc = orc.orc.topk_compress(K, LR, np.float32(mu or 0.0), keep, g, orc.m, orc.e, orc.sel,
                               orc.rank, orc.vals)
    assert rc == 0
    gs = TopkGpu(w, keep, mu=mu)
    wm = H.tensor_word_mask(off, n, d_pad)
    # the same inputs twice on one plan: the first call finds the threshold
    # outside the histogram window (it starts at the bottom of the key range),
    # the second one inside the window the first call placed
    for call in range(2):
        gs.e.copy_(torch.from_numpy(e))
        if momentum:
            gs.m.copy_(torch.from_numpy(m0))
        gs.saef.saef_topk_compress(gs.plan, K, float(LR), float(mu or 0.0), H.dev(g), gs.m, gs.e,
                                   gs.sel, gs.rank, gs.vals)
        torch.cuda.synchronize()
        H.assert_words_equal(H.host(gs.sel, np.uint64), orc.sel, wm, f"selection, call {call}")
        assert np.array_equal(_u32(gs.rank)[:, wm], orc.rank[:, wm]), f"rank words, call {call}"
        H.assert_f32_equal(H.host(gs.vals), orc.vals, np.ones(orc.vals.shape[-1], bool),
                           f"values, call {call}")
        got_e = H.host(gs.e)
        H.assert_f32_equal(got_e, orc.e, msk, f"errors, call {call}")
        assert np.isnan(got_e[:, ~msk]).all(), "padding written"
        if momentum:
            H.assert_f32_equal(H.host(gs.m), orc.m, msk, f"momentum buffers, call {call}")
    assert gs.status() == 0


@pytest.mark.parametrize("pct", [1, 3, 5])
@pytest.mark.parametrize("K", [3, 5, 12, 17])
@pytest.mark.parametrize("mode", [1, 0], ids=["dc", "sc"])
def test_topk_aggregate_parity(mode, K, pct):
    """Server step on oracle-made messages.  The server kernel reads the
    workers in batches of 8 (K <= 8) or 16: K = 3 and 12 leave part of a batch
    empty, K = 17 takes two batches; /K is not a power of two for 3, 5, 12, 17.
    Below 1/32 kept (1% and 3%) it gathers over the union of the workers' kept
    elements when one batch holds every worker (K <= 16; at 3%, K = 5 or 12,
    a pass holds more than 64 union elements) and per (worker, word) pair at
    K = 17; at 5% it takes one load per worker and batch."""
    w = W.custom(ADVERSARIAL + [200_000], K=K, scale_range=(1e-3, 1.0), seed=321, mode=mode)
    keep = W.topk_keep(w, pct)
    _case(f"topk aggregate mode={mode} K={K} pct={pct}")
    off, n, d_pad = w.layout()
    assert (int(keep.sum()) * 32 >= d_pad) == (pct == 5)  # which gather the server takes
    msk = W.tensor_mask(w)
    orc = TopkOracle(w, keep)
    g = W.gradients(w, 0)
    assert orc.orc.topk_compress(K, LR, 0.0, keep, g, None, orc.e, orc.sel, orc.rank,
                                 orc.vals) == 0
    rng = np.random.default_rng(9)
    es0 = (rng.standard_normal(d_pad) * 0.01).astype(np.float32)
    orc.e_srv[:] = es0
    avg = np.zeros(d_pad, np.float32)
    x0 = orc.x.copy()
    assert orc.orc.topk_aggregate(K, mode, keep, orc.sel, orc.vals, orc.x, orc.e_srv,
                                  orc.srv_sel, orc.srv_rank, orc.srv_vals, avg) == 0
    gs = TopkGpu(w, keep)
    sel = H.dev(orc.sel)
    rank = torch.from_numpy(orc.rank.view(np.int32)).cuda()
    vals = H.dev(orc.vals)
    gs.e_srv.copy_(torch.from_numpy(es0))
    gs.x.copy_(torch.from_numpy(x0))
    avg_d = torch.zeros(d_pad, dtype=torch.float32, device="cuda")
    gs.saef.saef_topk_aggregate(gs.plan, K, mode, sel, rank, vals, gs.x, gs.e_srv if mode else None,
                                gs.srv_sel if mode else None, gs.srv_rank if mode else None,
                                gs.srv_vals if mode else None, avg=avg_d)
    torch.cuda.synchronize()
    H.assert_f32_equal(H.host(avg_d), avg, msk, "mean")
    H.assert_f32_equal(H.host(gs.x), orc.x, msk, "weights")
    if mode == 1:
        wm = H.tensor_word_mask(off, n, d_pad)
        H.assert_words_equal(H.host(gs.srv_sel, np.uint64), orc.srv_sel, wm, "server selection")
        assert np.array_equal(_u32(gs.srv_rank)[wm], orc.srv_rank[wm])
        H.assert_f32_equal(H.host(gs.srv_vals), orc.srv_vals,
                           np.ones(orc.srv_vals.shape[-1], bool), "server values")
        H.assert_f32_equal(H.host(gs.e_srv), orc.e_srv, msk, "server error")
    assert gs.status() == 0


# data scale of successive calls on one plan: the threshold falls far below
# the histogram window placed by the previous call (the lowest bin), far
# above it (the bin above it), back inside it, then 4, 3, 10 and 5 binades
# down in turn (the one-binade bins below the window, 2 and 1 binades under
# it, and the lowest bin again) with jumps back up in between
SCALES = [1.0, 2.0 ** -20, 2.0 ** 30, 2.0 ** 30 * 1.5, 1.0, 2.0 ** -4, 2.0 ** -7, 1.0,
          2.0 ** -10, 2.0 ** -5, 1.0]


def test_topk_threshold_moves():
    """Successive compress and server calls on one plan whose data scale jumps
    by many binades: the kept set must not depend on where the previous
    call's threshold placed the histogram window."""
    K = 3
    w = W.custom([5000, 70001, 300_000], K=K, scale_range=(1e-2, 1.0), seed=77)
    keep = W.topk_keep(w, 1)
    off, n, d_pad = w.layout()
    msk = W.tensor_mask(w)
    wm = H.tensor_word_mask(off, n, d_pad)
    orc = TopkOracle(w, keep)
    gs = TopkGpu(w, keep)
    rng = np.random.default_rng(5)
    for c, scale in enumerate(SCALES):
        _case(f"topk threshold moves: call {c} scale {scale}")
        sc = np.float32(scale)
        g = (W.gradients(w, c) * sc).astype(np.float32)
        e = (rng.standard_normal((K, d_pad)) * np.float32(0.01) * sc).astype(np.float32)
        es = (rng.standard_normal(d_pad) * np.float32(0.01) * sc).astype(np.float32)
        orc.e[:] = e
        orc.e_srv[:] = es
        assert orc.orc.topk_compress(K, LR, 0.0, keep, g, None, orc.e, orc.sel, orc.rank,
                                     orc.vals) == 0
        assert orc.orc.topk_aggregate(K, 1, keep, orc.sel, orc.vals, orc.x, orc.e_srv,
                                      orc.srv_sel, orc.srv_rank, orc.srv_vals, None) == 0
        gs.e.copy_(torch.from_numpy(e))
        gs.e_srv.copy_(torch.from_numpy(es))
        gs.saef.saef_topk_compress(gs.plan, K, float(LR), 0.0, H.dev(g), None, gs.e, gs.sel,
                                   gs.rank, gs.vals)
        gs.saef.saef_topk_aggregate(gs.plan, K, 1, gs.sel, gs.rank, gs.vals, gs.x, gs.e_srv,
                                    gs.srv_sel, gs.srv_rank, gs.srv_vals)
        torch.cuda.synchronize()
        H.assert_words_equal(H.host(gs.sel, np.uint64), orc.sel, wm, f"selection, call {c}")
        assert np.array_equal(_u32(gs.rank)[:, wm], orc.rank[:, wm]), f"rank words, call {c}"
        H.assert_f32_equal(H.host(gs.vals), orc.vals, np.ones(orc.vals.shape[-1], bool),
                           f"values, call {c}")
        H.assert_f32_equal(H.host(gs.e), orc.e, msk, f"errors, call {c}")
        H.assert_words_equal(H.host(gs.srv_sel, np.uint64), orc.srv_sel, wm,
                             f"server selection, call {c}")
        H.assert_f32_equal(H.host(gs.srv_vals), orc.srv_vals,
                           np.ones(orc.srv_vals.shape[-1], bool), f"server values, call {c}")
        H.assert_f32_equal(H.host(gs.e_srv), orc.e_srv, msk, f"server error, call {c}")
        H.assert_f32_equal(H.host(gs.x), orc.x, msk, f"weights, call {c}")
    assert gs.status() == 0


# successive calls on one plan for the Delta pass's speculative lists (the
# elements just below the previous threshold and above): (data scale, hot
# tile).  A small drop of the threshold stays within the lists' bound, a
# larger one falls below it (Delta read again), a hot tile (its values x 8)
# overflows its list while the other tiles use theirs, and values of few
# distinct magnitudes overflow every list.
SPEC_CALLS = [(1.0, False), (1.0, False), (0.97, False), (1.0, False), (0.75, False),
              (1.0, True), (1.0, False), (1.0, "ties"), (1.0, False)]


def test_topk_speculative_lists():
    """Compress and server calls on one plan where the gather takes each
    tile from its speculative list or from Delta: bit-equal either way."""
    K = 3
    w = W.custom([5000, 70001, 300_000, 33], K=K, scale_range=(1e-2, 1.0), seed=91)
    keep = W.topk_keep(w, 1)
    off, n, d_pad = w.layout()
    msk = W.tensor_mask(w)
    wm = H.tensor_word_mask(off, n, d_pad)
    orc = TopkOracle(w, keep)
    gs = TopkGpu(w, keep)
    rng = np.random.default_rng(6)
    for c, (scale, hot) in enumerate(SPEC_CALLS):
        _case(f"topk speculative lists: call {c} scale {scale} hot {hot}")
        sc = np.float32(scale)
        g = (W.gradients(w, c % 2) * sc).astype(np.float32)
        e = (rng.standard_normal((K, d_pad)) * np.float32(0.01) * sc).astype(np.float32)
        if hot is True:
            a = int(off[1]) + 4096
            g[:, a:a + 2048] *= np.float32(8.0)
            e[:, a:a + 2048] *= np.float32(8.0)
        elif hot == "ties":
            g = _tie_values(rng, g.shape)
            e = np.zeros_like(e)
        e = np.where(msk, e, np.float32(0.0)).astype(np.float32)
        es = (rng.standard_normal(d_pad) * np.float32(0.01) * sc).astype(np.float32)
        es = np.where(msk, es, np.float32(0.0)).astype(np.float32)
        orc.e[:] = e
        orc.e_srv[:] = es
        assert orc.orc.topk_compress(K, LR, 0.0, keep, g, None, orc.e, orc.sel, orc.rank,
                                     orc.vals) == 0
        assert orc.orc.topk_aggregate(K, 1, keep, orc.sel, orc.vals, orc.x, orc.e_srv,
                                      orc.srv_sel, orc.srv_rank, orc.srv_vals, None) == 0
        gs.e.copy_(torch.from_numpy(e))
        gs.e_srv.copy_(torch.from_numpy(es))
        gs.saef.saef_topk_compress(gs.plan, K, float(LR), 0.0, H.dev(g), None, gs.e, gs.sel,
                                   gs.rank, gs.vals)
        gs.saef.saef_topk_aggregate(gs.plan, K, 1, gs.sel, gs.rank, gs.vals, gs.x, gs.e_srv,
                                    gs.srv_sel, gs.srv_rank, gs.srv_vals)
        torch.cuda.synchronize()
        H.assert_words_equal(H.host(gs.sel, np.uint64), orc.sel, wm, f"selection, call {c}")
        assert np.array_equal(_u32(gs.rank)[:, wm], orc.rank[:, wm]), f"rank words, call {c}"
        H.assert_f32_equal(H.host(gs.vals), orc.vals, np.ones(orc.vals.shape[-1], bool),
                           f"values, call {c}")
        H.assert_f32_equal(H.host(gs.e), orc.e, msk, f"errors, call {c}")
        H.assert_words_equal(H.host(gs.srv_sel, np.uint64), orc.srv_sel, wm,
                             f"server selection, call {c}")
        H.assert_f32_equal(H.host(gs.srv_vals), orc.srv_vals,
                           np.ones(orc.srv_vals.shape[-1], bool), f"server values, call {c}")
        H.assert_f32_equal(H.host(gs.e_srv), orc.e_srv, msk, f"server error, call {c}")
        H.assert_f32_equal(H.host(gs.x), orc.x, msk, f"weights, call {c}")
    assert gs.status() == 0


ROUND_CASES = {
    "resnet56_1pct_dc": (W.get("resnet56").with_(rounds=12, period=0), 1, None),
    "resnet56_10pct_avg": (W.get("resnet56").with_(rounds=12, period=4), 10, None),
    "resnet56_5pct_momentum": (W.get("resnet56").with_(rounds=8, period=0), 5, 0.9),
    "ragged_sc_avg": (W.custom(ADVERSARIAL + [70001], K=3, period=3, rounds=7, mode=0,
                               scale_range=(1e-4, 1e-1), dist="laplace_zeros", seed=998), 5, None),
    "flat64k_1pct": (W.get("flat64k"), 1, None),
}


@pytest.mark.parametrize("name", list(ROUND_CASES))
def test_topk_round_parity(name):
    """saef_topk_round over every iteration against the oracle."""
    w, pct, mu = ROUND_CASES[name]
    keep = W.topk_keep(w, pct)
    _case(f"topk round {name} K={w.K} L={w.L} rounds={w.rounds} pct={pct} mu={mu}")
    orc = TopkOracle(w, keep, mu=mu)
    gs = TopkGpu(w, keep, mu=mu)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        orc.round(t, g)
        gs.round(t, g)
        compare_topk(gs, orc, t, name, mode=w.mode)
    assert gs.status() == 0


HALVES_CASES = {
    "resnet56_5pct_avg_dc": (W.get("resnet56").with_(rounds=8, period=3), 5),
    "ragged_1pct_sc": (W.custom(ADVERSARIAL + [70001], K=3, period=0, rounds=6, mode=0,
                                scale_range=(1e-4, 1e-1), seed=991), 1),
}


@pytest.mark.parametrize("variant", [0, 1], ids=["ef", "saef"])
@pytest.mark.parametrize("name", list(HALVES_CASES))
def test_topk_round_halves_parity(name, variant):
    """Top-K in two halves (the EF branch of the paper's Table 1 comparison,
    and SAEF) with the mismatch bounds at every iteration."""
    w, pct = HALVES_CASES[name]
    keep = W.topk_keep(w, pct)
    _case(f"topk halves {name} variant={variant}")
    orc = TopkOracle(w, keep)
    gs = TopkGpu(w, keep)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        want = orc.begin(t, variant)
        got = gs.begin(t, variant)
        H.assert_mismatch_close(got, want, w, w.K, f"{name} t={t}")
        orc.end(g)
        gs.end(t, g)
        compare_topk(gs, orc, t, f"{name} v{variant}", mode=w.mode)
    assert gs.status() == 0


def test_topk_closed_loop_quadratic_ef_vs_saef():
    """Gradients taken at the evaluation point (noisy quadratic, fp32
    elementwise on both sides): with Top-K the EF and SAEF trajectories
    differ, and each matches the oracle bit for bit."""
    w = W.get("resnet56").with_(period=0, rounds=6)
    keep = W.topk_keep(w, 5)
    off, n, d_pad = w.layout()
    finals = []
    for variant in (0, 1):
        _case(f"topk closed loop variant={variant}")
        rng = np.random.default_rng(77)
        xstar = (rng.standard_normal(d_pad) * 0.05).astype(np.float32)
        xstar_d = torch.from_numpy(xstar).cuda()
        orc = TopkOracle(w, keep)
        gs = TopkGpu(w, keep)
        for t in range(w.rounds):
            noise = (rng.standard_normal((w.K, d_pad)) * 0.01).astype(np.float32)
            orc.begin(t, variant, mismatch=False)
            gs.begin(t, variant, mismatch=False)
            rows = orc.xh if variant == 1 else np.repeat(orc.xh[:1], w.K, axis=0)
            g_host = (np.float32(0.5) * (rows - xstar)).astype(np.float32) + noise
            xh_d = gs.xh if variant == 1 else gs.xh[:1].expand(w.K, d_pad)
            g_dev = (0.5 * (xh_d - xstar_d)) + torch.from_numpy(noise).cuda()
            orc.end(g_host)
            gs.end(t, g_dev.contiguous())
            compare_topk(gs, orc, t, f"closed loop v{variant}")
        finals.append(orc.x.copy())
    assert not np.array_equal(finals[0], finals[1])


def test_topk_invalid_and_range():
    w = W.custom([100, 7], K=2)
    from paper_2008_05823_amd import saef
    lay = saef.Layout(*w.layout(), 2)
    with pytest.raises(saef.SaefError):
        saef.TopK(lay, [0, 1])           # keep must be >= 1
    with pytest.raises(saef.SaefError):
        saef.TopK(lay, [101, 1])         # and <= n
    gs = TopkGpu(w, [3, 1])
    with pytest.raises(saef.SaefError):  # mu without a momentum buffer
        saef.saef_topk_compress(gs.plan, 2, 0.1, 0.9, gs.g, None, gs.e, gs.sel, gs.rank, gs.vals)
    g = torch.zeros_like(gs.g)
    g[1, 5] = float("inf")
    saef.saef_topk_compress(gs.plan, 2, 0.1, 0.0, g, None, gs.e, gs.sel, gs.rank, gs.vals)
    assert gs.status() == saef.ERANGE
    assert gs.status() == saef.OK        # the flag clears


def test_topk_graph_replay_parity():
    """saef_topk_round captured in HIP graphs (one per kind of iteration:
    t = 0 with plain errors, pending errors, pending errors with averaging),
    replayed with the gradients copied in between replays and checked
    against the oracle after every replay."""
    w = W.get("resnet56").with_(rounds=8, period=4)
    keep = W.topk_keep(w, 5)
    _case(f"topk graph replay resnet56 K={w.K} rounds={w.rounds}")
    orc = TopkOracle(w, keep)
    gs = TopkGpu(w, keep)
    S = gs.saef
    graphs = {}
    for t in range(w.rounds):
        kind = (t > 0, (t + 1) % w.period == 0)
        if kind not in graphs:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                S.saef_topk_round(gs.plan, t, w.period, gs.K, w.lr, 0.0, w.mode, gs.g, None, gs.e,
                                  gs.e_srv, gs.x, gs.xh, gs.sel, gs.rank, gs.vals, gs.srv_sel,
                                  gs.srv_rank, gs.srv_vals)
            graphs[kind] = graph
        grad = W.gradients(w, t)
        gs.g.copy_(torch.from_numpy(grad))
        graphs[kind].replay()
        torch.cuda.synchronize()
        orc.round(t, grad)
        compare_topk(gs, orc, t, "graph replay", mode=w.mode)
    assert len(graphs) == 3
    assert gs.status() == 0
