"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each pin_* function takes the path of a built oracle library and raises
AssertionError when the oracle disagrees with:
  - hand-derived worked examples of Eq. (2) and Algorithm 1 (tests/golden),
  - exact rational arithmetic (Python Fraction) on small random inputs,
  - closed forms and invariants: ||C(v)||_1 = ||v||_1, the delta-compressor
    equality, the auxiliary-variable identity Eq. (3) (Appendix A),
    zero error = scaled SignSGD, identical workers = one worker, p = 1.
The test module runs them on the real oracle; the mutation test runs them on
oracle builds with planted mistakes and expects each build to fail one.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from oracle import oracle as O
from tests import exact, golden_io

LR = np.float32(0.1)


def _one_tensor_layout(sizes):
    sizes = np.asarray(sizes, dtype=np.int64)
    padded = (sizes + 63) // 64 * 64
    off = np.concatenate([[0], np.cumsum(padded)[:-1]]).astype(np.int64)
    return off, sizes, int(padded.sum())


def _rand_values(rng, n, spread=True):
    """fp32 values with varied magnitudes, exact zeros of both signs and a few
    subnormals; all well inside the exact-sum range."""
    v = rng.standard_normal(n).astype(np.float32)
    if spread:
        v *= np.float32(2.0) ** rng.integers(-30, 6, n).astype(np.float32)
        pick = rng.random(n)
        v[pick < 0.05] = 0.0
        v[(pick >= 0.05) & (pick < 0.08)] = -0.0
        v[(pick >= 0.08) & (pick < 0.10)] = np.float32(3e-42) * np.sign(
            v[(pick >= 0.08) & (pick < 0.10)] + 0.5)
    return v


# ---------------------------------------------------------------- goldens

def pin_goldens(libpath):
    for name in golden_io.names():
        _run_golden(libpath, name)


def _run_topk_golden(libpath, name, gd):
    K = int(gd["K"][0])
    lr = np.float32(float(gd["lr"][0]))
    sizes = [int(s) for s in gd["sizes"]]
    keep = np.array([int(k) for k in gd["keep"]], np.int64)
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    W = d_pad // 64
    total = int(keep.sum())
    n0 = sizes[0]
    sel = np.zeros((K, W), np.uint64)
    rank = np.zeros((K, W), np.uint32)
    vals = np.zeros((K, total), np.float32)

    def vec(v):
        out = np.zeros(d_pad, np.float32)
        out[:len(v)] = golden_io.floats(v)
        return out

    if gd["op"][0] == "topk_compress":
        g = np.stack([vec(gd[f"g.{k}"]) for k in range(K)])
        e = np.stack([vec(gd[f"e.{k}"]) for k in range(K)])
        assert orc.topk_compress(K, lr, 0.0, keep, g, None, e, sel, rank, vals) == O.OK, name
    else:
        mode, period, rounds = int(gd["mode"][0]), int(gd["period"][0]), int(gd["rounds"][0])
        x = vec(gd["x0"])
        e = np.zeros((K, d_pad), np.float32)
        e_srv = np.zeros(d_pad, np.float32)
        xh = np.zeros((K, d_pad), np.float32)
        srv_sel = np.zeros(W, np.uint64)
        srv_rank = np.zeros(W, np.uint32)
        srv_vals = np.zeros(total, np.float32)
        for t in range(rounds):
            g = np.stack([vec(gd[f"g.{t}.{k}"]) for k in range(K)])
            rc = orc.topk_round(t, period, K, lr, 0.0, mode, keep, g, None, e, e_srv, x, xh, sel,
                                rank, vals, srv_sel, srv_rank, srv_vals)
            assert rc == O.OK, name
        assert np.array_equal(x[:n0], golden_io.floats(gd["expect.x"])), (name, x[:n0])
        if mode == 1:
            assert np.array_equal(srv_sel, golden_io.words(gd["expect.srv_words"])), name
            assert np.array_equal(srv_vals, golden_io.floats(gd["expect.srv_vals"])), name
            assert np.array_equal(e_srv[:n0], golden_io.floats(gd["expect.e_srv"])), name
    for k in range(K):
        assert np.array_equal(sel[k], golden_io.words(gd[f"expect.words.{k}"])), (name, k)
        assert np.array_equal(vals[k], golden_io.floats(gd[f"expect.vals.{k}"])), (name, k)
        assert np.array_equal(e[k, :n0], golden_io.floats(gd[f"expect.e.{k}"])), (name, k, e[k])
        if f"expect.xh.{k}" in gd:
            assert np.array_equal(xh[k, :n0], golden_io.floats(gd[f"expect.xh.{k}"])), (name, k)


def _run_golden(libpath, name):
    gd = golden_io.load(name)
    if gd["op"][0].startswith("topk"):
        return _run_topk_golden(libpath, name, gd)
    K = int(gd["K"][0])
    lr = np.float32(float(gd["lr"][0]))
    sizes = [int(s) for s in gd["sizes"]]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    L = len(sizes)
    W = d_pad // 64
    signs = np.zeros((K, W), np.uint64)
    scales = np.zeros((K, L), np.float32)

    def vec(vals):
        out = np.zeros(d_pad, np.float32)
        out[:len(vals)] = golden_io.floats(vals)
        return out

    if gd["op"][0] == "compress":
        g = np.stack([vec(gd[f"g.{k}"]) for k in range(K)])
        e = np.stack([vec(gd[f"e.{k}"]) for k in range(K)])
        assert orc.compress(K, lr, g, e, signs, scales) == O.OK, name
        xh = x = e_srv = srv_signs = srv_scales = None
    else:
        mode, period, rounds = int(gd["mode"][0]), int(gd["period"][0]), int(gd["rounds"][0])
        mu = np.float32(float(gd["mu"][0])) if "mu" in gd else None
        m = np.zeros((K, d_pad), np.float32)
        x = vec(gd["x0"])
        e = np.zeros((K, d_pad), np.float32)
        e_srv = np.zeros(d_pad, np.float32)
        xh = np.zeros((K, d_pad), np.float32)
        srv_signs = np.zeros(W, np.uint64)
        srv_scales = np.zeros(L, np.float32)
        variant = int(gd["variant"][0]) if "variant" in gd else None
        mism = np.zeros(2 * L, np.float64)
        for t in range(rounds):
            g = np.stack([vec(gd[f"g.{t}.{k}"]) for k in range(K)])
            if variant is not None:
                # the two halves of the iteration, with the mismatch bounds
                rc = orc.round_begin(t, period, K, mode, variant, e, e_srv, x, xh, mism)
                assert rc == O.OK, name
                rc = orc.round_end(K, lr, 0.0, mode, g, None, e, e_srv, x, signs, scales,
                                   srv_signs, srv_scales)
            elif mu is None:
                rc = orc.round(t, period, K, lr, mode, g, e, e_srv, x, xh, signs, scales,
                               srv_signs, srv_scales)
            else:
                rc = orc.round_momentum(t, period, K, lr, mu, mode, g, m, e, e_srv, x, xh, signs,
                                        scales, srv_signs, srv_scales)
            assert rc == O.OK, name
        if "expect.mismatch_ef" in gd:
            assert np.array_equal(mism[:L], golden_io.floats(gd["expect.mismatch_ef"])), (name, mism)
            assert np.array_equal(mism[L:], golden_io.floats(gd["expect.mismatch_saef"])), (name,
                                                                                             mism)
    n0 = sizes[0]
    exp_scales = golden_io.floats(gd["expect.scales"])
    assert np.array_equal(scales.reshape(-1), exp_scales), (name, scales, exp_scales)
    for k in range(K):
        assert np.array_equal(signs[k], golden_io.words(gd[f"expect.words.{k}"])), (name, k)
        assert np.array_equal(e[k, :n0], golden_io.floats(gd[f"expect.e.{k}"])), (name, k, e[k])
        if f"expect.xh.{k}" in gd:
            assert np.array_equal(xh[k, :n0], golden_io.floats(gd[f"expect.xh.{k}"])), (name, k)
        if f"expect.m.{k}" in gd:
            assert np.array_equal(m[k, :n0], golden_io.floats(gd[f"expect.m.{k}"])), (name, k)
    if "expect.x" in gd:
        assert np.array_equal(x[:n0], golden_io.floats(gd["expect.x"])), (name, x)
    if "expect.srv_scales" in gd:
        assert np.array_equal(srv_scales, golden_io.floats(gd["expect.srv_scales"])), name
        assert np.array_equal(srv_signs, golden_io.words(gd["expect.srv_words"])), name
        assert np.array_equal(e_srv[:n0], golden_io.floats(gd["expect.e_srv"])), name


# ---------------------------------------------------------------- exact steps

def _bit(words, off, i):
    return int((int(words[off // 64 + i // 64]) >> (i % 64)) & 1)


def _check_scale(s, values):
    """s within half an fp32 ulp (plus the binary64 steps and the 2^-80
    quantum) of the exact mean absolute value."""
    exact_mean = sum(abs(exact.frac(v)) for v in values) / len(values)
    err = abs(Fraction(float(s)) - exact_mean)
    bound = Fraction(exact.ulp32(s)) / 2 + exact_mean * Fraction(1, 2**51) + Fraction(1, 2**80)
    assert err <= bound, (float(s), float(exact_mean))


def pin_compress_exact(libpath, seed=1):
    rng = np.random.default_rng(seed)
    sizes = [1, 3, 64, 65, 130, 7]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L = 3, len(sizes)
    g = np.full((K, d_pad), np.nan, np.float32)    # NaN poison on padding
    e = np.full((K, d_pad), np.nan, np.float32)
    for l in range(L):
        g[:, off[l]:off[l] + n[l]] = _rand_values(rng, K * n[l]).reshape(K, n[l])
        e[:, off[l]:off[l] + n[l]] = _rand_values(rng, K * n[l]).reshape(K, n[l]) * 0.01
    e0 = e.copy()
    signs = np.full((K, d_pad // 64), 0xFFFF, np.uint64)
    scales = np.zeros((K, L), np.float32)
    assert orc.compress(K, LR, g, e, signs, scales) == O.OK
    for k in range(K):
        for l in range(L):
            o, nl = int(off[l]), int(n[l])
            p = [exact.rn32(Fraction(float(LR)) * exact.frac(g[k, o + i]) + exact.frac(e0[k, o + i]))
                 for i in range(nl)]
            _check_scale(scales[k, l], p)
            s = Fraction(float(scales[k, l]))
            for i in range(nl):
                bit = _bit(signs[k], o, i)
                assert bit == (1 if p[i] >= 0 else 0), (k, l, i)
                c = s if bit else -s
                assert e[k, o + i] == exact.rn32(exact.frac(p[i]) - c), (k, l, i)
            nw = (nl + 63) // 64
            last = int(signs[k, o // 64 + nw - 1])
            if nl % 64:
                assert last >> (nl % 64) == 0, "bits past the tensor end must be 0"
        pad = ~_tensor_mask(off, n, d_pad)
        assert np.isnan(e[k, pad]).all(), "padding must not be written"


def _tensor_mask(off, n, d_pad):
    m = np.zeros(d_pad, bool)
    for o, nl in zip(off, n):
        m[o:o + nl] = True
    return m


def pin_aggregate_exact(libpath, seed=2):
    """K = 4: the binary64 sum of four +-scale values of similar size is exact,
    so the mean is the fp32 rounding of the exact mean."""
    rng = np.random.default_rng(seed)
    sizes = [5, 70]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L, W = 4, len(sizes), d_pad // 64
    for mode in (1, 0):
        signs = rng.integers(0, 2**64, (K, W), dtype=np.uint64)
        for l in range(L):  # bits past the tensor end are 0 in a valid message
            o, nl = int(off[l]), int(n[l])
            last = o // 64 + (nl - 1) // 64
            if nl % 64:
                signs[:, last] &= np.uint64((1 << (nl % 64)) - 1)
        scales = (rng.random((K, L)) + 0.5).astype(np.float32)
        x = rng.standard_normal(d_pad).astype(np.float32)
        e_srv = (rng.standard_normal(d_pad) * 0.1).astype(np.float32)
        x0, es0 = x.copy(), e_srv.copy()
        avg = np.zeros(d_pad, np.float32)
        srv_signs = np.zeros(W, np.uint64)
        srv_scales = np.zeros(L, np.float32)
        rc = orc.aggregate(K, mode, signs, scales, x, e_srv, srv_signs, srv_scales, avg)
        assert rc == O.OK
        for l in range(L):
            o, nl = int(off[l]), int(n[l])
            delta = []
            for i in range(nl):
                msg = [Fraction(float(scales[k, l])) * (1 if _bit(signs[k], o, i) else -1)
                       for k in range(K)]
                a = exact.rn32(sum(msg) / K)
                assert avg[o + i] == a, (mode, l, i)
                if mode == 1:
                    delta.append(exact.rn32(exact.frac(es0[o + i]) + exact.frac(a)))
                else:
                    assert x[o + i] == exact.rn32(exact.frac(x0[o + i]) - exact.frac(a))
            if mode == 1:
                _check_scale(srv_scales[l], delta)
                s = Fraction(float(srv_scales[l]))
                for i in range(nl):
                    bit = _bit(srv_signs, o, i)
                    assert bit == (1 if delta[i] >= 0 else 0)
                    c = s if bit else -s
                    assert e_srv[o + i] == exact.rn32(exact.frac(delta[i]) - c)
                    assert x[o + i] == exact.rn32(exact.frac(x0[o + i]) - c)


def pin_step_ahead_and_average_exact(libpath, seed=3):
    rng = np.random.default_rng(seed)
    sizes = [9, 64]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    for K in (1, 2, 4, 3):
        x = rng.standard_normal(d_pad).astype(np.float32)
        e = (rng.standard_normal((K, d_pad)) * 0.3).astype(np.float32)
        xh = np.zeros((K, d_pad), np.float32)
        assert orc.step_ahead(K, x, e, xh) == O.OK
        m = _tensor_mask(off, n, d_pad)
        for k in range(K):
            for j in np.nonzero(m)[0]:
                assert xh[k, j] == exact.rn32(exact.frac(x[j]) - exact.frac(e[k, j]))
        e0 = e.copy()
        assert orc.error_average(K, e) == O.OK
        for j in np.nonzero(m)[0]:
            mean = sum(exact.frac(e0[k, j]) for k in range(K)) / K
            want = exact.rn32(mean)
            if K & (K - 1) == 0:
                assert all(e[k, j] == want for k in range(K)), (K, j)
            else:  # binary64 division by 3 rounds once before fp32
                assert all(abs(Fraction(float(e[k, j])) - mean) <=
                           Fraction(exact.ulp32(want)) / 2 * (1 + Fraction(1, 2**28))
                           for k in range(K))
                assert len({float(e[k, j]) for k in range(K)}) == 1


# ---------------------------------------------------------------- invariants

def run_rounds(libpath, w, rounds, gens=None):
    """Run the oracle over `rounds` iterations of workload w; returns the
    per-round states needed by the invariants."""
    from paper_2008_05823_amd import workloads as W
    off, n, d_pad = w.layout()
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L = w.K, w.L
    x = W.initial_x(w)
    e = np.zeros((K, d_pad), np.float32)
    e_srv = np.zeros(d_pad, np.float32)
    xh = np.zeros((K, d_pad), np.float32)
    signs = np.zeros((K, d_pad // 64), np.uint64)
    scales = np.zeros((K, L), np.float32)
    srv_signs = np.zeros(d_pad // 64, np.uint64)
    srv_scales = np.zeros(L, np.float32)
    hist = []
    for t in range(rounds):
        g = W.gradients(w, t) if gens is None else gens(t)
        rc = orc.round(t, w.period, K, np.float32(w.lr), w.mode, g, e, e_srv, x, xh,
                       signs, scales, srv_signs, srv_scales)
        assert rc == O.OK
        hist.append(dict(g=g, x=x.copy(), e=e.copy(), e_srv=e_srv.copy(), xh=xh.copy(),
                         signs=signs.copy(), scales=scales.copy(),
                         srv_signs=srv_signs.copy(), srv_scales=srv_scales.copy()))
    return hist


def pin_auxiliary_identity(libpath):
    """Eq. (3) / Appendix A: x~_t = x_t - (e_t + mean_k e^(k)_t) moves by
    -lr * mean_k g^(k)_t each iteration, whatever the compressor does, in both
    compression modes and with error averaging (which keeps mean_k e^(k))."""
    from paper_2008_05823_amd import workloads as W
    for mode, period in ((1, 0), (1, 2), (0, 3)):
        w = W.custom([100, 64, 1, 300], K=3, period=period, rounds=6, mode=mode,
                     scale_range=(1e-3, 1.0), seed=77 + mode + period)
        hist = run_rounds(libpath, w, w.rounds)
        x0 = W.initial_x(w).astype(np.float64)
        m = W.tensor_mask(w)
        drift = np.zeros_like(x0)
        mag = np.abs(x0).copy()
        for h in hist:
            drift += np.float64(w.lr) * h["g"].astype(np.float64).mean(axis=0)
            mag += np.abs(h["x"]) + np.abs(h["e_srv"]) + np.abs(h["e"]).mean(axis=0) + \
                np.float64(w.lr) * np.abs(h["g"]).mean(axis=0)
        h = hist[-1]
        xt = h["x"].astype(np.float64) - (h["e_srv"].astype(np.float64) +
                                          h["e"].astype(np.float64).mean(axis=0))
        err = np.abs(xt - (x0 - drift))[m]
        tol = 8 * 2.0 ** -24 * mag[m] + 1e-30
        assert (err <= tol).all(), (mode, period, float(err.max()))


def pin_delta_compressor_equality(libpath, seed=4):
    """Assumption (delta-approximate compressor): for C of Eq. (2) the bound is
    an equality, ||v - C(v)||^2 = ||v||^2 - ||v||_1^2 / d."""
    rng = np.random.default_rng(seed)
    sizes = [1000, 333, 64]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K = 2
    g = np.zeros((K, d_pad), np.float32)
    for l in range(len(sizes)):
        g[:, off[l]:off[l] + n[l]] = rng.laplace(size=(K, n[l])).astype(np.float32)
    e = np.zeros((K, d_pad), np.float32)
    signs = np.zeros((K, d_pad // 64), np.uint64)
    scales = np.zeros((K, len(sizes)), np.float32)
    p = np.stack([np.float32(LR) * g[k] for k in range(K)]).astype(np.float32)
    assert orc.compress(K, LR, g, e, signs, scales) == O.OK
    for k in range(K):
        for l in range(len(sizes)):
            sl = slice(off[l], off[l] + n[l])
            v = p[k, sl].astype(np.float64)
            lhs = np.sum(e[k, sl].astype(np.float64) ** 2)
            rhs = np.sum(v ** 2) - np.sum(np.abs(v)) ** 2 / n[l]
            assert abs(lhs - rhs) <= 1e-5 * np.sum(v ** 2), (k, l, lhs, rhs)
            # ||C(v)||_1 = d * scale equals ||v||_1
            assert abs(n[l] * np.float64(scales[k, l]) - np.sum(np.abs(v))) <= \
                2 ** -22 * np.sum(np.abs(v))


def pin_zero_error_is_scaled_signsgd(libpath, seed=5):
    """With e = 0, K = 1, single-way and no averaging, one iteration is
    scaled SignSGD: x_1 = x_0 - mean|lr g| * sign(g)."""
    rng = np.random.default_rng(seed)
    sizes = [200, 1]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    g = rng.standard_normal((1, d_pad)).astype(np.float32)
    g[0, 3] = 0.0
    x = rng.standard_normal(d_pad).astype(np.float32)
    x0 = x.copy()
    e = np.zeros((1, d_pad), np.float32)
    xh = np.zeros((1, d_pad), np.float32)
    signs = np.zeros((1, d_pad // 64), np.uint64)
    scales = np.zeros((1, 2), np.float32)
    rc = orc.round(0, 0, 1, LR, 0, g, e, None, x, xh, signs, scales, None, None)
    assert rc == O.OK
    for l in range(2):
        sl = slice(off[l], off[l] + n[l])
        lrg = (np.float32(LR) * g[0, sl]).astype(np.float32)
        s = np.mean(np.abs(lrg.astype(np.float64)))
        assert abs(np.float64(scales[0, l]) - s) <= 2 ** -23 * s
        sign = np.where(g[0, sl] >= 0, 1.0, -1.0).astype(np.float32)
        want = (x0[sl] - scales[0, l] * sign).astype(np.float32)
        assert np.array_equal(x[sl], want)
        assert np.array_equal(xh[0, sl], x0[sl])


def pin_identical_workers(libpath):
    """K identical workers give exactly the single-worker iteration."""
    from paper_2008_05823_amd import workloads as W
    base = W.custom([129, 64, 3], K=1, period=2, rounds=4, scale_range=(0.01, 1.0), seed=91)
    one = run_rounds(libpath, base, 4)
    for K in (2, 4):
        wk = base.with_(K=K)
        many = run_rounds(libpath, wk, 4,
                          gens=lambda t: np.repeat(W.gradients(base, t), K, axis=0))
        for a, b in zip(one, many):
            assert np.array_equal(a["x"], b["x"]) and np.array_equal(a["e_srv"], b["e_srv"])
            for k in range(K):
                assert np.array_equal(a["e"][0], b["e"][k])
                assert np.array_equal(a["xh"][0], b["xh"][k])
                assert np.array_equal(a["signs"][0], b["signs"][k])


def pin_period_one(libpath):
    """p = 1: errors are averaged before every step ahead, so every worker
    evaluates its gradient at the same point."""
    from paper_2008_05823_amd import workloads as W
    w = W.custom([77, 128], K=3, period=1, rounds=4, scale_range=(0.1, 1.0), seed=5)
    for h in run_rounds(libpath, w, 4):
        for k in range(1, w.K):
            assert np.array_equal(h["xh"][0], h["xh"][k])


def pin_l1_fixed_exact(libpath, seed=11):
    """The exact L1 sum equals the Python big-integer sum of floor(|v| 2^80)."""
    import ctypes
    lib = O.lib(libpath)
    rng = np.random.default_rng(seed)
    for trial in range(10):
        v = _rand_values(rng, int(rng.integers(1, 2000)))
        if trial == 0:
            v[:3] = [np.float32(524287.97), -np.float32(2.0 ** -80), np.float32(1.5 * 2 ** -80)]
        hi, lo = ctypes.c_uint64(), ctypes.c_uint64()
        rc = lib.oracle_l1_fixed(v.ctypes.data, v.size, ctypes.byref(hi), ctypes.byref(lo))
        assert rc == O.OK
        assert (hi.value << 64) | lo.value == exact.exact_l1_fixed(v)


def pin_momentum_exact(libpath, seed=12):
    """m' is the fp32 rounding of mu m + g, Delta that of eta m' + e; mu = 0
    with m = 0 gives exactly the plain worker step."""
    rng = np.random.default_rng(seed)
    sizes = [70, 3]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L = 2, len(sizes)
    mu = np.float32(0.9)
    g = (rng.standard_normal((K, d_pad)) * 0.5).astype(np.float32)
    m = (rng.standard_normal((K, d_pad)) * 0.3).astype(np.float32)
    e = (rng.standard_normal((K, d_pad)) * 0.01).astype(np.float32)
    m0, e0 = m.copy(), e.copy()
    signs = np.zeros((K, d_pad // 64), np.uint64)
    scales = np.zeros((K, L), np.float32)
    assert orc.compress_momentum(K, LR, mu, g, m, e, signs, scales) == O.OK
    for k in range(K):
        for l in range(L):
            o, nl = int(off[l]), int(n[l])
            p = []
            for i in range(nl):
                mm = exact.rn32(Fraction(float(mu)) * exact.frac(m0[k, o + i]) +
                                exact.frac(g[k, o + i]))
                assert m[k, o + i] == mm, (k, l, i)
                p.append(exact.rn32(Fraction(float(LR)) * exact.frac(mm) +
                                    exact.frac(e0[k, o + i])))
            _check_scale(scales[k, l], p)
            s = Fraction(float(scales[k, l]))
            for i in range(nl):
                c = s if _bit(signs[k], o, i) else -s
                assert e[k, o + i] == exact.rn32(exact.frac(p[i]) - c), (k, l, i)
    # mu = 0 and m = 0: the same as the plain worker step
    e1, e2 = e0.copy(), e0.copy()
    s1, s2 = np.zeros_like(signs), np.zeros_like(signs)
    c1, c2 = np.zeros_like(scales), np.zeros_like(scales)
    mz = np.zeros_like(m)
    assert orc.compress_momentum(K, LR, np.float32(0.0), g, mz, e1, s1, c1) == O.OK
    assert orc.compress(K, LR, g, e2, s2, c2) == O.OK
    assert np.array_equal(e1, e2) and np.array_equal(s1, s2) and np.array_equal(c1, c2)
    msk = _tensor_mask(off, n, d_pad)
    assert np.array_equal(mz[:, msk], g[:, msk])


def pin_auxiliary_identity_momentum(libpath):
    """Eq. (3) / Appendix A with momentum: x~ moves by -(eta/K) sum_k m^(k)_{t+1}."""
    from paper_2008_05823_amd import workloads as W
    for mode, period in ((1, 0), (1, 3), (0, 0)):
        w = W.custom([90, 64, 5], K=3, period=period, rounds=6, mode=mode,
                     scale_range=(1e-2, 1.0), seed=31 + mode + period)
        off, n, d_pad = w.layout()
        orc = O.Oracle(off, n, d_pad, libpath)
        K, L = w.K, w.L
        mu = np.float32(0.9)
        x0 = W.initial_x(w)
        x = x0.copy()
        m = np.zeros((K, d_pad), np.float32)
        e = np.zeros((K, d_pad), np.float32)
        e_srv = np.zeros(d_pad, np.float32)
        xh = np.zeros((K, d_pad), np.float32)
        signs = np.zeros((K, d_pad // 64), np.uint64)
        scales = np.zeros((K, L), np.float32)
        ss = np.zeros(d_pad // 64, np.uint64)
        sc = np.zeros(L, np.float32)
        drift = np.zeros(d_pad)
        mag = np.abs(x0).astype(np.float64)
        for t in range(w.rounds):
            g = W.gradients(w, t)
            rc = orc.round_momentum(t, period, K, np.float32(w.lr), mu, mode, g, m, e, e_srv, x,
                                    xh, signs, scales, ss, sc)
            assert rc == O.OK
            drift += np.float64(w.lr) * m.astype(np.float64).mean(axis=0)
            mag += np.abs(x) + np.abs(e_srv) + np.abs(e).mean(axis=0) + \
                np.float64(w.lr) * np.abs(m).mean(axis=0)
        xt = x.astype(np.float64) - (e_srv.astype(np.float64) + e.astype(np.float64).mean(axis=0))
        msk = W.tensor_mask(w)
        err = np.abs(xt - (x0.astype(np.float64) - drift))[msk]
        assert (err <= 8 * 2.0 ** -24 * mag[msk] + 1e-30).all(), (mode, period, float(err.max()))


def run_split_rounds(libpath, w, rounds, variant, gens=None):
    """Run the two halves of each iteration (round_begin with the mismatch
    bounds, round_end) over `rounds` iterations of workload w; records the
    state seen by the bounds (after averaging) and the end state."""
    from paper_2008_05823_amd import workloads as W
    off, n, d_pad = w.layout()
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L = w.K, w.L
    x = W.initial_x(w)
    e = np.zeros((K, d_pad), np.float32)
    e_srv = np.zeros(d_pad, np.float32)
    xh = np.zeros((K, d_pad), np.float32)
    signs = np.zeros((K, d_pad // 64), np.uint64)
    scales = np.zeros((K, L), np.float32)
    srv_signs = np.zeros(d_pad // 64, np.uint64)
    srv_scales = np.zeros(L, np.float32)
    hist = []
    for t in range(rounds):
        g = W.gradients(w, t) if gens is None else gens(t)
        mism = np.full(2 * L, np.nan)
        x_start = x.copy()
        assert orc.round_begin(t, w.period, K, w.mode, variant, e, e_srv, x, xh, mism) == O.OK
        seen = dict(e=e.copy(), e_srv=e_srv.copy(), x=x_start)
        assert orc.round_end(K, np.float32(w.lr), 0.0, w.mode, g, None, e, e_srv, x, signs,
                             scales, srv_signs, srv_scales) == O.OK
        hist.append(dict(g=g, mism=mism, seen=seen, xh=xh.copy(), x=x.copy(), e=e.copy(),
                         e_srv=e_srv.copy(), signs=signs.copy(), scales=scales.copy(),
                         srv_signs=srv_signs.copy(), srv_scales=srv_scales.copy()))
    return hist


def _per_tensor(v, off, n):
    return np.array([v[..., o:o + m].sum() for o, m in zip(off, n)])


def pin_mismatch_identities(libpath):
    """The two bounds against identities that hold in exact arithmetic:
    (1/K) sum_k ||u - e^(k)||^2 = ||e_srv||^2 + (1/K) sum_k ||ebar - e^(k)||^2
    (the cross term vanishes because sum_k (ebar - e^(k)) = 0), and
    ||u||^2 = SAEF bound + 2 <u, ebar> - (1/K) sum_k ||e^(k)||^2; at an
    averaging iteration the step-ahead bound is the server error alone,
    ||e_t||^2 (zero in single-way compression) -- the "Error Averaging" bound."""
    from paper_2008_05823_amd import workloads as W
    cases = [W.custom([300, 64, 1, 129], K=3, period=3, rounds=6, scale_range=(1e-3, 1.0),
                      seed=31),
             W.custom([1000, 17], K=4, period=2, rounds=4, mode=0, scale_range=(0.01, 1.0),
                      seed=32, dist="laplace_zeros")]
    for w in cases:
        off, n, _ = w.layout()
        for t, h in enumerate(run_split_rounds(libpath, w, w.rounds, variant=1)):
            e = h["seen"]["e"].astype(np.float64)
            es = h["seen"]["e_srv"].astype(np.float64) if w.mode == 1 else 0.0 * e[0]
            ebar = e.mean(axis=0)
            u = es + ebar
            ef, sa = h["mism"][:w.L], h["mism"][w.L:]
            srv2 = _per_tensor(es * es, off, n)
            var = _per_tensor(((ebar - e) ** 2).mean(axis=0), off, n)
            np.testing.assert_allclose(sa, srv2 + var, rtol=1e-12, atol=1e-300)
            cross = _per_tensor(u * ebar, off, n)
            ek2 = _per_tensor((e * e).mean(axis=0), off, n)
            scale = ef + sa + 2 * np.abs(cross) + ek2
            assert np.all(np.abs(ef - (sa + 2 * cross - ek2)) <= 1e-12 * scale), (t, ef)
            if (t + 1) % w.period == 0:
                if w.mode == 0:
                    assert np.all(sa == 0.0), (t, sa)
                else:
                    np.testing.assert_allclose(sa, srv2, rtol=1e-12)


def pin_mismatch_proposition(libpath):
    """Proposition of the "Step Ahead" section, single-way (no server error):
    for the same local errors the step-ahead bound is the smaller one exactly
    when the spread of the errors across workers is at most the squared norm
    of their mean."""
    rng = np.random.default_rng(33)
    off, n, d_pad = _one_tensor_layout([500])
    orc = O.Oracle(off, n, d_pad, libpath)
    K = 5
    seen = set()
    for trial in range(40):
        c = rng.standard_normal(500).astype(np.float32)
        spread = np.float32(10.0 ** rng.uniform(-2, 1))
        e = np.zeros((K, d_pad), np.float32)
        e[:, :500] = c + spread * rng.standard_normal((K, 500)).astype(np.float32)
        ef, sa = orc.mismatch(K, e)
        e64 = e[:, :500].astype(np.float64)
        var = ((e64 - e64.mean(axis=0)) ** 2).sum() / K
        mean2 = (e64.mean(axis=0) ** 2).sum()
        assert (sa[0] <= ef[0]) == (var <= mean2), (trial, sa, ef, var, mean2)
        seen.add(bool(var <= mean2))
    assert seen == {True, False}


def pin_ef_variant(libpath):
    """Local error feedback (the EF branch) takes the gradient at x_t itself;
    both branches form Delta^(k) = e^(k) + eta m^(k) (Algorithm 1), so with
    gradients that do not depend on the evaluation point the two branches
    produce the same state, bit for bit, and only the evaluation points
    differ: x_t for EF, x_t - e^(k)_t for SAEF."""
    from paper_2008_05823_amd import workloads as W
    w = W.custom([200, 64, 3], K=3, period=3, rounds=5, scale_range=(0.01, 1.0), seed=34)
    ef = run_split_rounds(libpath, w, w.rounds, variant=0)
    sa = run_split_rounds(libpath, w, w.rounds, variant=1)
    for a, b in zip(ef, sa):
        for key in ("x", "e", "e_srv", "signs", "scales", "srv_signs", "srv_scales"):
            assert np.array_equal(a[key], b[key]), key
        np.testing.assert_array_equal(a["mism"], b["mism"])
        assert np.array_equal(a["xh"][0], a["seen"]["x"])
        for k in range(w.K):
            exp = (b["seen"]["x"] - b["seen"]["e"][k]).astype(np.float32)
            assert np.array_equal(b["xh"][k], exp)


# ---------------------------------------------------------------- Top-K

def _topk_message_dense(sel_row, rank_row, vals_row, off, n, keep):
    """C(v) of every tensor decoded through the rank words (the oracle itself
    decodes by walking the bits in order)."""
    out = {}
    voff = 0
    for l in range(len(n)):
        o, nl = int(off[l]), int(n[l])
        c = np.zeros(nl, np.float32)
        kept = np.zeros(nl, bool)
        for i in range(nl):
            w = o // 64 + i // 64
            word = int(sel_row[w])
            if (word >> (i % 64)) & 1:
                below = bin(word & ((1 << (i % 64)) - 1)).count("1")
                c[i] = vals_row[voff + int(rank_row[w]) + below]
                kept[i] = True
        out[l] = (c, kept)
        voff += int(keep[l])
    return out


def _topk_values(rng, n):
    """Values with repeated magnitudes (ties), zeros of both signs and spread."""
    v = _rand_values(rng, n)
    dup = rng.random(n) < 0.2
    v[dup] = np.float32(0.375) * np.where(rng.random(int(dup.sum())) < 0.5, 1, -1)
    return v


def pin_topk_compress_exact(libpath, seed=41):
    """Top-K worker step against the definition's properties: exactly k_l
    kept, every kept magnitude >= every dropped one, equal magnitudes at the
    cut kept in index order, Delta = fma(lr, g, e) rounded once (checked in
    exact arithmetic), e = Delta - C(Delta) exactly, the rank words count the
    kept elements before each word, padding untouched."""
    rng = np.random.default_rng(seed)
    sizes = [1, 3, 64, 65, 130, 200]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L = 3, len(sizes)
    for keep in ([1, 1, 1, 1, 1, 1], [1, 2, 7, 64, 13, 100], [1, 3, 64, 65, 130, 200]):
        keep = np.array(keep, np.int64)
        g = np.full((K, d_pad), np.nan, np.float32)
        e = np.full((K, d_pad), np.nan, np.float32)
        for l in range(L):
            g[:, off[l]:off[l] + n[l]] = _topk_values(rng, K * n[l]).reshape(K, n[l])
            e[:, off[l]:off[l] + n[l]] = _topk_values(rng, K * n[l]).reshape(K, n[l]) * 0.01
        e0 = e.copy()
        sel = np.full((K, d_pad // 64), 0xFFFF, np.uint64)
        rank = np.zeros((K, d_pad // 64), np.uint32)
        vals = np.zeros((K, int(keep.sum())), np.float32)
        assert orc.topk_compress(K, LR, 0.0, keep, g, None, e, sel, rank, vals) == O.OK
        for k in range(K):
            dec = _topk_message_dense(sel[k], rank[k], vals[k], off, n, keep)
            for l in range(L):
                o, nl = int(off[l]), int(n[l])
                p = np.array([exact.rn32(Fraction(float(LR)) * exact.frac(g[k, o + i])
                                         + exact.frac(e0[k, o + i])) for i in range(nl)],
                             np.float32)
                c, kept = dec[l]
                assert kept.sum() == keep[l], (k, l)
                mag = np.abs(p.astype(np.float64))
                if kept.sum() < nl:
                    lo_kept = mag[kept].min()
                    assert mag[~kept].max() <= lo_kept, (k, l)
                    ties_dropped = np.where(~kept & (mag == lo_kept))[0]
                    ties_kept = np.where(kept & (mag == lo_kept))[0]
                    if len(ties_dropped):
                        assert ties_kept.max() < ties_dropped.min(), (k, l)
                assert np.array_equal(c[kept], p[kept]), (k, l)
                err = e[k, o:o + nl]
                assert np.array_equal(err[kept], np.zeros(int(kept.sum()), np.float32))
                # (values: the exact reference does not carry the sign of a zero)
                assert np.array_equal(err[~kept], p[~kept])
                nw = (nl + 63) // 64
                if nl % 64:
                    assert int(sel[k, o // 64 + nw - 1]) >> (nl % 64) == 0
            pad = ~_tensor_mask(off, n, d_pad)
            assert np.isnan(e[k, pad]).all(), "padding must not be written"


def pin_topk_momentum_exact(libpath, seed=45):
    """Top-K worker step with momentum (Algorithm 1): m <- mu m + g and Delta =
    e + eta m, each rounded once (exact arithmetic); the message carries the
    kept Delta values."""
    rng = np.random.default_rng(seed)
    sizes = [100, 3]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K = 2
    keep = np.array([10, 2], np.int64)
    mu = np.float32(0.9)
    g = np.zeros((K, d_pad), np.float32)
    m = np.zeros((K, d_pad), np.float32)
    e = np.zeros((K, d_pad), np.float32)
    for l in range(2):
        sl = slice(int(off[l]), int(off[l] + n[l]))
        g[:, sl] = _topk_values(rng, K * int(n[l])).reshape(K, -1)
        m[:, sl] = _topk_values(rng, K * int(n[l])).reshape(K, -1)
        e[:, sl] = _topk_values(rng, K * int(n[l])).reshape(K, -1) * 0.01
    m0, e0 = m.copy(), e.copy()
    sel = np.zeros((K, d_pad // 64), np.uint64)
    rank = np.zeros((K, d_pad // 64), np.uint32)
    vals = np.zeros((K, int(keep.sum())), np.float32)
    assert orc.topk_compress(K, LR, mu, keep, g, m, e, sel, rank, vals) == O.OK
    for k in range(K):
        dec = _topk_message_dense(sel[k], rank[k], vals[k], off, n, keep)
        for l in range(2):
            o, nl = int(off[l]), int(n[l])
            mm = np.array([exact.rn32(exact.frac(mu) * exact.frac(m0[k, o + i])
                                      + exact.frac(g[k, o + i])) for i in range(nl)], np.float32)
            assert np.array_equal(m[k, o:o + nl], mm), (k, l)
            p = np.array([exact.rn32(exact.frac(LR) * exact.frac(mm[i])
                                     + exact.frac(e0[k, o + i])) for i in range(nl)], np.float32)
            c, kept = dec[l]
            assert np.array_equal(c[kept], p[kept]) and np.array_equal(e[k, o:o + nl][~kept],
                                                                       p[~kept]), (k, l)


def pin_topk_delta_compressor(libpath, seed=42):
    """Top-K is a delta-approximate compressor (the paper's compressor
    assumption) with delta = k_l / n_l per tensor:
    ||C(v) - v||^2 <= (1 - k_l/n_l) ||v||^2, in exact arithmetic."""
    rng = np.random.default_rng(seed)
    sizes = [5, 100, 257]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    for trial in range(6):
        keep = np.array([int(rng.integers(1, m + 1)) for m in sizes], np.int64)
        g = np.zeros((1, d_pad), np.float32)
        for l in range(len(sizes)):
            g[0, off[l]:off[l] + n[l]] = _topk_values(rng, int(n[l]))
        e = np.zeros_like(g)
        sel = np.zeros((1, d_pad // 64), np.uint64)
        rank = np.zeros((1, d_pad // 64), np.uint32)
        vals = np.zeros((1, int(keep.sum())), np.float32)
        assert orc.topk_compress(1, np.float32(1.0), 0.0, keep, g, None, e, sel, rank, vals) == 0
        for l in range(len(sizes)):
            o, nl = int(off[l]), int(n[l])
            v = [exact.frac(x) for x in g[0, o:o + nl]]
            r = [exact.frac(x) for x in e[0, o:o + nl]]   # v - C(v)
            lhs = sum(x * x for x in r)
            rhs = (1 - Fraction(int(keep[l]), nl)) * sum(x * x for x in v)
            assert lhs <= rhs, (trial, l)


def pin_topk_aggregate_exact(libpath, seed=43):
    """Top-K server step: the mean of the decoded messages is the correctly
    rounded binary64 worker-order sum / K (checked exactly when no binary64
    rounding can occur: K = 4 and values of a few bits), Delta = fp32(e_srv +
    mean), and the server message/error/x follow the Top-K definition; x
    changes only at kept elements (x - Delta there)."""
    rng = np.random.default_rng(seed)
    sizes = [70, 129]
    off, n, d_pad = _one_tensor_layout(sizes)
    orc = O.Oracle(off, n, d_pad, libpath)
    K, L = 4, 2
    keep = np.array([9, 40], np.int64)
    total = int(keep.sum())
    g = np.zeros((K, d_pad), np.float32)
    for l in range(L):
        g[:, off[l]:off[l] + n[l]] = (rng.integers(-64, 65, (K, int(n[l]))) / 16.0)
    e = np.zeros_like(g)
    sel = np.zeros((K, d_pad // 64), np.uint64)
    rank = np.zeros((K, d_pad // 64), np.uint32)
    vals = np.zeros((K, total), np.float32)
    assert orc.topk_compress(K, np.float32(1.0), 0.0, keep, g, None, e, sel, rank, vals) == 0
    for mode in (0, 1):
        x = (rng.integers(-100, 101, d_pad) / 8.0).astype(np.float32)
        x0 = x.copy()
        e_srv = (rng.integers(-8, 9, d_pad) / 32.0).astype(np.float32)
        es0 = e_srv.copy()
        avg = np.zeros(d_pad, np.float32)
        ss = np.zeros(d_pad // 64, np.uint64)
        sr = np.zeros(d_pad // 64, np.uint32)
        sv = np.zeros(total, np.float32)
        assert orc.topk_aggregate(K, mode, keep, sel, vals, x, e_srv, ss, sr, sv, avg) == 0
        decs = [_topk_message_dense(sel[k], rank[k], vals[k], off, n, keep) for k in range(K)]
        for l in range(L):
            o, nl = int(off[l]), int(n[l])
            mean = [exact.rn32(sum((exact.frac(decs[k][l][0][i]) for k in range(K)), Fraction(0))
                               / K) for i in range(nl)]
            assert np.array_equal(avg[o:o + nl], np.array(mean, np.float32)), (mode, l)
            if mode == 0:
                want = [exact.rn32(exact.frac(x0[o + i]) - exact.frac(mean[i])) for i in range(nl)]
                assert np.array_equal(x[o:o + nl], np.array(want, np.float32))
                continue
            D = np.array([exact.rn32(exact.frac(es0[o + i]) + exact.frac(mean[i]))
                          for i in range(nl)], np.float32)
            c, kept = _topk_message_dense(ss, sr, sv, off, n, keep)[l]
            assert kept.sum() == keep[l]
            mag = np.abs(D.astype(np.float64))
            if kept.sum() < nl:
                assert mag[~kept].max() <= mag[kept].min()
            assert np.array_equal(c[kept], D[kept])
            assert np.array_equal(e_srv[o:o + nl][kept], np.zeros(int(kept.sum()), np.float32))
            assert np.array_equal(e_srv[o:o + nl][~kept], D[~kept])
            want_x = np.where(kept, [exact.rn32(exact.frac(x0[o + i]) - exact.frac(D[i]))
                                     for i in range(nl)], x0[o:o + nl]).astype(np.float32)
            assert np.array_equal(x[o:o + nl], want_x)


def pin_topk_auxiliary_identity(libpath):
    """Eq. (3) for any compressor: x~_T = x_T - (e_srv + mean_k e^(k)) =
    x_0 - eta sum_t mean_k g_t (binary64 with a rounding allowance), with
    Top-K in both modes and with averaging; keep = n gives plain SGD (no
    error at all)."""
    from paper_2008_05823_amd import workloads as W
    for mode, period, pct in ((1, 0, 10), (0, 3, 5), (1, 2, 1), (1, 0, 100)):
        w = W.custom([300, 64, 1, 129], K=3, period=period, rounds=5, mode=mode,
                     scale_range=(1e-3, 1.0), seed=44 + pct)
        off, n, d_pad = w.layout()
        keep = W.topk_keep(w, pct)
        orc = O.Oracle(off, n, d_pad, libpath)
        K, L = w.K, w.L
        x = W.initial_x(w)
        x0 = x.astype(np.float64)
        e = np.zeros((K, d_pad), np.float32)
        e_srv = np.zeros(d_pad, np.float32)
        xh = np.zeros((K, d_pad), np.float32)
        sel = np.zeros((K, d_pad // 64), np.uint64)
        rank = np.zeros((K, d_pad // 64), np.uint32)
        vals = np.zeros((K, int(keep.sum())), np.float32)
        ss = np.zeros(d_pad // 64, np.uint64)
        sr = np.zeros(d_pad // 64, np.uint32)
        sv = np.zeros(int(keep.sum()), np.float32)
        gsum = np.zeros(d_pad)
        mag = np.zeros(d_pad)
        for t in range(w.rounds):
            g = W.gradients(w, t)
            assert orc.topk_round(t, period, K, np.float32(w.lr), 0.0, mode, keep, g, None, e,
                                  e_srv, x, xh, sel, rank, vals, ss, sr, sv) == O.OK
            gsum += g.astype(np.float64).mean(axis=0)
            mag += np.abs(g.astype(np.float64)).mean(axis=0) * w.lr
        m = W.tensor_mask(w)
        xt = x.astype(np.float64) - (e_srv.astype(np.float64) * (mode == 1)
                                     + e.astype(np.float64).mean(axis=0))
        want = x0 - np.float64(np.float32(w.lr)) * gsum
        tol = 16 * w.rounds * 2.0 ** -24 * (np.abs(x0) + mag + np.abs(xt)) + 1e-30
        assert np.all(np.abs(xt - want)[m] <= tol[m]), (mode, period, pct)
        if pct == 100:
            assert not e[:, m].any() and not e_srv[m].any()


QUICK_PINS = [pin_goldens, pin_topk_compress_exact, pin_topk_momentum_exact,
              pin_topk_delta_compressor,
              pin_topk_aggregate_exact, pin_topk_auxiliary_identity, pin_mismatch_identities, pin_mismatch_proposition, pin_ef_variant, pin_momentum_exact, pin_auxiliary_identity_momentum, pin_l1_fixed_exact, pin_compress_exact, pin_aggregate_exact,
              pin_step_ahead_and_average_exact, pin_auxiliary_identity,
              pin_delta_compressor_equality, pin_zero_error_is_scaled_signsgd,
              pin_identical_workers, pin_period_one]
