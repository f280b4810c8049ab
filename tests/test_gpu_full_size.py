"""Parity at the full workload sizes, in the launch configuration bench.py
times (saef_round over the whole tensor list, same tiles and kernels).

The scaled-sign workloads are compared with the oracle in full: every tensor,
every element, every iteration of the workload (ResNet-50: 161 tensors, 20
iterations; BERT-base: 199 tensors, K = 16, 10 iterations; one tensor of
2^28 elements, K = 8, 5 iterations), including the server error, the
weights and the server message.  The oracle runs piecewise on a thread pool
(tests.split_oracle; its equality with the whole-layout oracle is a CPU
test), which brings a ResNet-50 iteration to about a second of host time.

A mid-size multi-tensor layout of more than 2048 tiles covers the long
XCD tile runs of the step-ahead and averaging kernels with the pending
corrections, over several iterations that include error averaging.

The Top-K workloads (the paper's second compressor) are checked on a sample
of tensors (the largest included) and by the defining properties of Top-K.

Gradient recipe at these sizes: iteration t uses the seeded gradient set of
t mod 2 (two sets, as in bench.py), so the host generates 2 K vectors.
"""
import numpy as np
import pytest
import torch

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H
from tests.split_oracle import SplitOracle, default_threads, rows_equal

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _log(msg):
    print(f"[full-size] {msg}", flush=True)


def _sub_workload(w, idx):
    """The same workload restricted to the tensors idx (packed layout)."""
    tensors = tuple(w.tensors[i] for i in idx)
    return w.with_(tensors=tensors, name=w.name + "_sample")


def _gather(full, off, n, idx, sub_off, sub_dpad):
    """Copy tensor slices of a (..., d_pad) host array into the packed layout."""
    out = np.zeros(full.shape[:-1] + (sub_dpad,), full.dtype)
    for j, i in enumerate(idx):
        out[..., sub_off[j]:sub_off[j] + n[i]] = full[..., off[i]:off[i] + n[i]]
    return out


def _gather_words(full, off, n, idx, sub_off, sub_w):
    out = np.zeros(full.shape[:-1] + (sub_w,), full.dtype)
    for j, i in enumerate(idx):
        nw = (n[i] + 63) // 64
        out[..., sub_off[j] // 64:sub_off[j] // 64 + nw] = full[..., off[i] // 64:off[i] // 64 + nw]
    return out


def _device_slices(t, off, n, idx):
    """Download only the sampled tensors of a device (..., d_pad) tensor."""
    parts = [t[..., off[i]:off[i] + n[i]].cpu().numpy() for i in idx]
    return parts


def compare_full(gpu: dict, so: SplitOracle, t: int, tag: str):
    """Every element, word and scale of the state against the oracle, bit for
    bit (padding included: neither side ever writes it, both start at 0)."""
    names = ["signs", "e", "xh", "x"] + (["srv_signs", "e_srv"] if so.w.mode == 1 else [])
    for name in names:
        if not rows_equal(gpu[name], getattr(so, name)):
            so.m = None
            H.compare_state(gpu, so, t, tag)  # names the first difference
            raise AssertionError(f"{tag} t={t}: {name} differs from the oracle")
    if not np.array_equal(gpu["scales"].view(np.uint32), so.scales.view(np.uint32)):
        so.m = None
        H.compare_state(gpu, so, t, tag)
        raise AssertionError(f"{tag} t={t}: worker scales differ")
    if so.w.mode == 1 and not np.array_equal(gpu["srv_scales"].view(np.uint32),
                                             so.srv_scales.view(np.uint32)):
        raise AssertionError(f"{tag} t={t}: server scales differ")


def run_full(w: W.Workload, rounds: int, tag: str):
    """rounds iterations of w through saef_round, each compared in full."""
    threads = default_threads()
    _log(f"{tag}: K={w.K} L={w.L} d={w.d} d_pad={w.d_pad}, {rounds} iterations, period "
         f"{w.period}, oracle on {threads} threads")
    grads = [W.gradients(w, s, threads=threads) for s in range(min(2, rounds))]
    _log(f"{tag}: gradients generated")
    so = SplitOracle(w, threads=threads)
    gs = H.GpuState(w)
    g_dev = [torch.from_numpy(g).cuda() for g in grads]
    for t in range(rounds):
        gs.round(t, g_dev[t % 2])
        so.round(t, grads[t % 2])
        compare_full(gs.plain(), so, t, tag)
        _log(f"{tag}: iteration {t} matches the oracle on every element"
             + (" (error averaging)" if w.period and (t + 1) % w.period == 0 else ""))
    assert gs.status() == 0


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["resnet50", "bert_base"])
def test_full_size_every_tensor(name):
    """ResNet-50 (K = 8, 20 iterations, averaging at t = 19) and BERT-base
    (K = 16, 10 iterations, averaging at t = 4 and 9): the whole state after
    every iteration."""
    w = W.get(name)
    run_full(w, w.rounds, name)


@pytest.mark.timeout(900)
def test_full_size_flat256m():
    """One tensor of 2^28 elements, K = 8, 5 iterations (averaging at t = 4):
    the whole state after every iteration, server error, weights and server
    message included."""
    w = W.get("flat256m")
    run_full(w, w.rounds, "flat256m")


def _mid_size_workload():
    """48 tensors of seeded sizes (1 .. 300000, ragged), more than 2048 tiles."""
    rng = np.random.default_rng(2048)
    sizes = np.concatenate([rng.integers(1, 300001, 40), rng.integers(1, 200, 6), [1, 64]])
    return W.custom(sizes.tolist(), K=8, period=3, rounds=7, dist="laplace_zeros",
                    scale_range=(1e-5, 1e-2), seed=W.SEED_BASE + 2048, name="mid")


@pytest.mark.timeout(600)
def test_mid_size_long_tile_runs():
    """A multi-tensor layout past 2048 tiles (the step-ahead and averaging
    kernels then deal runs of 64 tiles to each XCD) with the pending
    corrections, 7 iterations with averaging at t = 2 and 5, in full."""
    from paper_2008_05823_amd import saef
    w = _mid_size_workload()
    lay = saef.Layout(*w.layout(), w.K)
    n_tiles = lay.info()["n_tiles"]
    lay.close()
    assert n_tiles >= 2048, n_tiles
    run_full(w, w.rounds, f"mid ({n_tiles} tiles)")


# conv1, bn1.bias, layer1.0.conv2, layer3.5.conv3, layer4.0.conv2 (the largest,
# 3x3x512x512), layer4.2.bn3.weight, fc.weight (2048x1000), fc.bias
TOPK_SAMPLE = ["conv1.weight", "bn1.bias", "layer1.0.conv2.weight", "layer3.5.conv3.weight",
               "layer4.0.conv2.weight", "layer4.2.bn3.weight", "fc.weight", "fc.bias"]


@pytest.mark.timeout(600)
def test_full_size_topk_resnet50():
    """Layer-wise Top-1% at the full ResNet-50 shape, K = 8, in the launch
    configuration bench.py --topk 1 times: saef_topk_round over the whole
    tensor list; the oracle runs the sampled tensors (the largest included)
    with the same gradient slices, bit for bit, for 4 iterations (averaging
    period 2 so that an averaging iteration is covered)."""
    from tests.test_gpu_topk import TopkGpu, TopkOracle, _u32
    w = W.get("resnet50").with_(period=2)
    names = [t for t, _ in w.tensors]
    idx = [names.index(s) for s in TOPK_SAMPLE]
    off, n, d_pad = w.layout()
    sw = _sub_workload(w, idx)
    s_off, s_n, s_dpad = sw.layout()
    keep = W.topk_keep(w, 1)
    rounds = 4
    _log(f"topk resnet50: K={w.K} L={w.L} d={w.d}, {rounds} iterations, oracle on {len(idx)} "
         f"tensors ({int(s_n.sum())} elements)")
    grads = [W.gradients(w, s, threads=default_threads()) for s in range(2)]
    x0 = W.initial_x(w)
    orc = TopkOracle(sw, keep[idx], x0=_gather(x0, off, n, idx, s_off, s_dpad))
    gs = TopkGpu(w, keep, x0=x0)
    g_dev = [torch.from_numpy(g).cuda() for g in grads]
    voff = np.concatenate([[0], np.cumsum(keep)[:-1]])
    for t in range(rounds):
        orc.round(t, _gather(grads[t % 2], off, n, idx, s_off, s_dpad))
        gs.round(t, g_dev[t % 2])
        torch.cuda.synchronize()

        def pack(dev_t):
            parts = _device_slices(dev_t, off, n, idx)
            out = np.zeros(dev_t.shape[:-1] + (s_dpad,), np.float32)
            for j, p in enumerate(parts):
                out[..., s_off[j]:s_off[j] + s_n[j]] = p
            return out
        m = W.tensor_mask(sw)
        wm = H.tensor_word_mask(s_off, s_n, s_dpad)
        tag = f"topk resnet50 t={t}"
        H.assert_f32_equal(pack(gs.plain_e()), orc.e, m, f"{tag} e")
        H.assert_f32_equal(pack(gs.xh), orc.xh, m, f"{tag} xh")
        H.assert_f32_equal(pack(gs.x), orc.x, m, f"{tag} weights")
        H.assert_f32_equal(pack(gs.e_srv), orc.e_srv, m, f"{tag} server error")
        sel = _gather_words(H.host(gs.sel, np.uint64), off, n, idx, s_off, s_dpad // 64)
        H.assert_words_equal(sel, orc.sel, wm, f"{tag} worker selection")
        rank = _gather_words(_u32(gs.rank), off, n, idx, s_off, s_dpad // 64)
        assert np.array_equal(rank[:, wm], orc.rank[:, wm]), f"{tag} worker rank words"
        ssel = _gather_words(H.host(gs.srv_sel, np.uint64), off, n, idx, s_off, s_dpad // 64)
        H.assert_words_equal(ssel, orc.srv_sel, wm, f"{tag} server selection")
        vals = H.host(gs.vals)
        svals = H.host(gs.srv_vals)
        o_voff = np.concatenate([[0], np.cumsum(keep[idx])[:-1]])
        for j, i in enumerate(idx):
            kl = int(keep[i])
            got = vals[:, voff[i]:voff[i] + kl]
            H.assert_f32_equal(got, orc.vals[:, o_voff[j]:o_voff[j] + kl], np.ones(kl, bool),
                               f"{tag} worker values of {names[i]}")
            H.assert_f32_equal(svals[voff[i]:voff[i] + kl], orc.srv_vals[o_voff[j]:o_voff[j] + kl],
                               np.ones(kl, bool), f"{tag} server values of {names[i]}")
        _log(f"topk resnet50: iteration {t} matches the oracle on the sampled tensors")
    assert gs.status() == 0


def _check_topk_row(delta, sel_words, vals, kept_count, tag):
    """Properties that define the Top-K of one vector, at any size: exactly
    kept_count kept, every kept magnitude >= every dropped one, equal
    magnitudes at the cut kept by lower index, the values in index order."""
    n = delta.size
    bits = np.unpackbits(sel_words.view(np.uint8), bitorder="little")[:n].astype(bool)
    assert int(bits.sum()) == kept_count, (tag, int(bits.sum()), kept_count)
    mag = np.abs(delta)
    lo_kept = mag[bits].min()
    if kept_count < n:
        hi_drop = mag[~bits].max()
        assert lo_kept >= hi_drop, (tag, lo_kept, hi_drop)
        if lo_kept == hi_drop:
            tie = mag == lo_kept
            assert np.flatnonzero(tie & bits).max() < np.flatnonzero(tie & ~bits).min(), tag
    assert np.array_equal(vals[:kept_count].view(np.uint32), delta[bits].view(np.uint32)), tag
    return bits


@pytest.mark.timeout(600)
def test_full_size_topk_flat256m():
    """Top-1% of one 2^28-element tensor (131072 tiles: 2048 tile groups in
    32 super-groups), K = 8, iteration 0 of saef_topk_round, checked
    against the defining properties of Top-K on every worker and on the
    server, and the error / weight updates bit for bit."""
    from tests.test_gpu_topk import TopkGpu
    w = W.get("flat256m")
    K = w.K
    keep = W.topk_keep(w, 1)
    k1 = int(keep[0])
    _log(f"topk flat256m: K={K} d={w.d} keep={k1}")
    g = W.gradients(w, 0, threads=default_threads())
    x0 = W.initial_x(w)
    gs = TopkGpu(w, keep, x0=x0)
    gs.round(0, torch.from_numpy(g).cuda())
    torch.cuda.synchronize()
    assert gs.status() == 0
    n = w.d
    lr = np.float32(w.lr)
    acc = np.zeros(n, np.float64)
    for k in range(K):
        # Delta = fma(lr, g, e) with e = +0: the exact product rounded once, and
        # a zero product becomes +0 (+0 + -0 = +0)
        delta = (np.float64(lr) * g[k, :n].astype(np.float64) + 0.0).astype(np.float32)
        sel = gs.sel[k].cpu().numpy().view(np.uint64)
        vals = gs.vals[k].cpu().numpy()
        bits = _check_topk_row(delta, sel, vals, k1, f"worker {k}")
        # saef_topk_round leaves the kept elements pending: e holds Delta
        # everywhere, and the plain error is 0 where bits are set
        e = gs.e[k, :n].cpu().numpy()
        want = delta
        bad = np.flatnonzero(e.view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, (f"worker {k} error: {bad.size} differ, first {bad[:5].tolist()}, "
                               f"got {e[bad[:5]].tolist()} want {want[bad[:5]].tolist()} "
                               f"kept {bits[bad[:5]].tolist()}")
        dense = np.zeros(n, np.float32)
        dense[bits] = delta[bits]
        acc += dense
        del delta, sel, vals, bits, e, want, dense
        _log(f"topk flat256m: worker {k} satisfies the Top-K properties")
    mean = (acc / K).astype(np.float32)
    del acc
    D = (np.float32(0.0) + mean).astype(np.float32)  # e_srv = 0 at t = 0
    bits = _check_topk_row(D, gs.srv_sel.cpu().numpy().view(np.uint64), gs.srv_vals.cpu().numpy(),
                           k1, "server")
    es = gs.e_srv[:n].cpu().numpy()
    want_es = np.where(bits, np.float32(0.0), D)
    bad = np.flatnonzero(es.view(np.uint32) != want_es.view(np.uint32))
    assert bad.size == 0, (f"server error: {bad.size} differ, first {bad[:5].tolist()}, "
                           f"got {es[bad[:5]].tolist()} want {want_es[bad[:5]].tolist()}")
    x = gs.x[:n].cpu().numpy()
    want_x = np.where(bits, (x0[:n] - D).astype(np.float32), x0[:n])
    bad = np.flatnonzero(x.view(np.uint32) != want_x.view(np.uint32))
    assert bad.size == 0, (f"weights: {bad.size} differ, first {bad[:5].tolist()}, "
                           f"got {x[bad[:5]].tolist()} want {want_x[bad[:5]].tolist()}")
    _log("topk flat256m: server and weights satisfy the Top-K properties")
