"""Parity at the full workload sizes, in the launch configuration bench.py
times (saef_round over the whole tensor list, same tiles and kernels).

The oracle cannot redo a whole ResNet-50 or BERT-base iteration for K workers
in test time, but it does not need to: every tensor evolves independently of
the others (one scale per tensor, everything else elementwise), so the oracle
runs the full iteration sequence on a sample of tensors -- the largest ones
included -- fed with the same gradient slices, and the GPU state of those
tensors must match it bit for bit after every iteration.

The 2^28-element single tensor is checked against one full oracle iteration
and, for later iterations, against properties that hold at any size.

Gradient recipe at these sizes: iteration t uses the seeded gradient set of
t mod 2 (two sets, as in bench.py), so the host generates 2 K vectors.
"""
import numpy as np
import pytest
import torch

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H

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


SAMPLES = {
    # conv1, bn1.bias, layer1.0.conv2, layer3.5.conv3, layer4.0.conv2 (the largest,
    # 3x3x512x512), layer4.2.bn3.weight, fc.weight (2048x1000), fc.bias
    "resnet50": ("resnet50", None, ["conv1.weight", "bn1.bias", "layer1.0.conv2.weight",
                                    "layer3.5.conv3.weight", "layer4.0.conv2.weight",
                                    "layer4.2.bn3.weight", "fc.weight", "fc.bias"]),
    # word embedding (largest, 30522x768), token type, a LayerNorm bias, a query
    # weight, an FFN input bias, the pooler bias; 5 iterations cover the
    # pending-correction path and the averaging iteration t = 4
    "bert_base": ("bert_base", 5, ["embeddings.word", "embeddings.token_type",
                                   "layer0.attn.ln.bias", "layer5.attn.query.weight",
                                   "layer11.ffn.in.bias", "pooler.bias"]),
}


@pytest.mark.parametrize("case", list(SAMPLES))
def test_full_size_sampled_tensors(case):
    name, rounds, sample_names = SAMPLES[case]
    w = W.get(name)
    rounds = rounds or w.rounds
    names = [t for t, _ in w.tensors]
    idx = [names.index(s) for s in sample_names]
    off, n, d_pad = w.layout()
    sw = _sub_workload(w, idx)
    s_off, s_n, s_dpad = sw.layout()
    _log(f"{case}: K={w.K} L={w.L} d={w.d}, {rounds} iterations, oracle on {len(idx)} tensors "
         f"({int(s_n.sum())} elements)")

    grads = [W.gradients(w, s) for s in range(2)]
    _log("gradients generated")
    x0 = W.initial_x(w)
    orc = H.OracleState(sw, x0=_gather(x0, off, n, idx, s_off, s_dpad))
    gs = H.GpuState(w, x0=x0)
    g_dev = [torch.from_numpy(g).cuda() for g in grads]
    f32 = dict(dtype=torch.float32, device="cuda")
    e_out = torch.empty((w.K, d_pad), **f32)
    es_out = torch.empty(d_pad, **f32)
    x_out = torch.empty(d_pad, **f32)
    for t in range(rounds):
        orc.round(t, _gather(grads[t % 2], off, n, idx, s_off, s_dpad))
        gs.round(t, g_dev[t % 2])
        gs.saef.saef_materialize(gs.layout, w.K, w.mode, gs.e, gs.e_srv, gs.x, gs.signs,
                                 gs.scales, gs.srv_signs, gs.srv_scales, e_out, es_out, x_out)
        torch.cuda.synchronize()
        # pack each state array tensor by tensor into the sample layout
        def pack(dev_t):
            parts = _device_slices(dev_t, off, n, idx)
            out = np.zeros(dev_t.shape[:-1] + (s_dpad,), np.float32)
            for j, p in enumerate(parts):
                out[..., s_off[j]:s_off[j] + s_n[j]] = p
            return out
        got = {"e": pack(e_out), "e_srv": pack(es_out), "x": pack(x_out), "xh": pack(gs.xh)}
        signs = H.host(gs.signs, np.uint64)
        got["signs"] = _gather_words(signs, off, n, idx, s_off, s_dpad // 64)
        got["srv_signs"] = _gather_words(H.host(gs.srv_signs, np.uint64), off, n, idx, s_off,
                                         s_dpad // 64)
        got["scales"] = H.host(gs.scales)[:, idx]
        got["srv_scales"] = H.host(gs.srv_scales)[idx]
        H.compare_state(got, orc, t, case)
        _log(f"{case}: iteration {t} matches the oracle on the sampled tensors")
    assert gs.status() == 0


def test_full_size_flat256m():
    """One tensor of 2^28 elements, K = 8: iteration 0 against the full oracle,
    later iterations against size-independent properties of Eq. (2)."""
    w = W.get("flat256m")
    off, n, d_pad = w.layout()
    K = w.K
    _log(f"flat256m: K={K} d={w.d}")
    grads = [W.gradients(w, s) for s in range(2)]
    x0 = W.initial_x(w)
    _log("gradients generated")
    gs = H.GpuState(w, x0=x0)
    g_dev = [torch.from_numpy(g).cuda() for g in grads]

    # iteration 0: full oracle, bit for bit
    orc = H.OracleState(w, x0=x0)
    orc.round(0, grads[0])
    _log("oracle iteration 0 done")
    gs.round(0, g_dev[0])
    H.compare_state(gs.plain(), orc, 0, "flat256m")
    _log("iteration 0 matches the oracle")
    del orc

    lr = np.float64(np.float32(w.lr))
    rng = np.random.default_rng(5)
    probe = rng.integers(0, w.d, 1 << 20)
    for t in range(1, w.rounds):
        check = t in (1, w.period - 1)  # first pending-correction iteration, averaging iteration
        prev = gs.plain() if check else None
        gs.round(t, g_dev[t % 2])
        if not check:
            continue
        cur = gs.plain()
        g = grads[t % 2]
        if (t + 1) % w.period == 0:
            # every worker starts from the binary64 mean of the errors (worker order), in fp32
            acc = np.zeros(w.d, np.float64)
            for k in range(K):
                acc += prev["e"][k]
            e_avg = (acc / K).astype(np.float32)
        for k in range(K):
            e_in = e_avg if (t + 1) % w.period == 0 else prev["e"][k]
            p = lr * g[k].astype(np.float64) + e_in.astype(np.float64)  # Delta, before rounding
            # sign words: bit i is [Delta_i >= 0] (rounding to fp32 keeps the sign)
            bits = np.packbits((p >= 0).astype(np.uint8), bitorder="little").view(np.uint64)
            assert np.array_equal(bits, cur["signs"][k]), (t, k)
            # ||C(Delta)||_1 = ||Delta||_1: n * scale is the L1 norm of Delta
            pf = p.astype(np.float32)
            l1 = np.abs(pf.astype(np.float64)).sum()
            assert abs(float(cur["scales"][k, 0]) * w.d - l1) <= 1e-6 * l1, (t, k)
            # e = Delta - C(Delta), on a probe of elements
            pp = pf[probe]
            s = cur["scales"][k, 0]
            want = (pp - np.where(pp >= 0, s, -s)).astype(np.float32)
            np.testing.assert_allclose(cur["e"][k][probe], want, rtol=1e-6, atol=1e-7)
            # step-ahead weights x_t - e_t
            xe = (prev["x"][probe] - e_in[probe]).astype(np.float32)
            np.testing.assert_allclose(cur["xh"][k][probe], xe, rtol=1e-6, atol=1e-7)
            del p, pf, bits
        _log(f"iteration {t} satisfies the size-independent checks")
    assert gs.status() == 0


def test_full_size_topk_resnet50():
    """Layer-wise Top-1% at the full ResNet-50 shape, K = 8, in the launch
    configuration bench.py --topk 1 times: saef_topk_round over the whole
    tensor list; the oracle runs the sampled tensors (the largest included)
    with the same gradient slices, bit for bit, for 4 iterations (averaging
    period 2 so that an averaging iteration is covered)."""
    from tests.test_gpu_topk import TopkGpu, TopkOracle, _u32
    w = W.get("resnet50").with_(period=2)
    names = [t for t, _ in w.tensors]
    idx = [names.index(s) for s in SAMPLES["resnet50"][2]]
    off, n, d_pad = w.layout()
    sw = _sub_workload(w, idx)
    s_off, s_n, s_dpad = sw.layout()
    keep = W.topk_keep(w, 1)
    rounds = 4
    _log(f"topk resnet50: K={w.K} L={w.L} d={w.d}, {rounds} iterations, oracle on {len(idx)} "
         f"tensors ({int(s_n.sum())} elements)")
    grads = [W.gradients(w, s) for s in range(2)]
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
    g = W.gradients(w, 0)
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
