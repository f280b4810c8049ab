"""Parity of the HIP library with the CPU oracle (needs an MI355X).

Every test runs the library through its C ABI (ctypes binding) on seeded
synthetic inputs and compares with the oracle on the same inputs: sign words
bit for bit, fp32 values bit for bit (which implies the 1e-6 relative /
1e-7 absolute acceptance bound).
"""
import numpy as np
import pytest
import torch

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H

pytestmark = pytest.mark.gpu

LR = np.float32(0.1)

# sizes around the wave (64), workgroup tile (4096) and word boundaries
ADVERSARIAL = [1, 3, 4, 10, 63, 64, 65, 255, 256, 257, 4095, 4096, 4097, 8193, 12345]


def _case(msg):
    print(f"[case] {msg}", flush=True)


def _rand_err(rng, K, w, scale=0.01):
    off, n, d_pad = w.layout()
    e = np.zeros((K, d_pad), np.float32)
    for o, nl in zip(off, n):
        e[:, o:o + nl] = rng.standard_normal((K, nl)).astype(np.float32) * np.float32(scale)
    return e


@pytest.mark.parametrize("K,sizes", [
    (1, [1]),
    (3, ADVERSARIAL),
    (8, [4096 * 3 + 17, 64, 1, 70000]),
    (4, [(1 << 20) + 3]),
    (2, [9_000_001, 64]),   # > 4096 tiles in one tensor: two-level scale reduction
])
def test_compress_parity(K, sizes):
    _case(f"compress K={K} sizes={sizes}")
    rng = np.random.default_rng(len(sizes) * 100 + K)
    w = W.custom(sizes, K=K, scale_range=(1e-3, 1.0), seed=K + 7)
    off, n, d_pad = w.layout()
    m = W.tensor_mask(w)
    g = W.gradients(w, 0)
    e = _rand_err(rng, K, w)
    e[:, ~m] = np.nan          # padding must stay untouched
    g[:, ~m] = np.nan
    orc = H.OracleState(w)
    orc.e[:] = e
    assert orc.orc.compress(K, LR, g, orc.e, orc.signs, orc.scales) == 0

    gs = H.GpuState(w)
    gs.e.copy_(torch.from_numpy(e))
    gd = H.dev(g)
    gs.saef.saef_compress(gs.layout, K, float(LR), gd, gs.e, gs.signs, gs.scales)
    got_e = H.host(gs.e)
    assert gs.status() == 0
    H.assert_words_equal(H.host(gs.signs, np.uint64), orc.signs,
                         H.tensor_word_mask(off, n, d_pad), "signs")
    H.assert_f32_equal(H.host(gs.scales), orc.scales, np.ones(w.L, bool), "scales")
    H.assert_f32_equal(got_e, orc.e, m, "errors")
    assert np.isnan(got_e[:, ~m]).all(), "padding was written"


@pytest.mark.parametrize("mode", [1, 0])
@pytest.mark.parametrize("K", [1, 3, 8, 16])
def test_aggregate_parity(mode, K):
    _case(f"aggregate mode={mode} K={K}")
    rng = np.random.default_rng(K * 10 + mode)
    w = W.custom([5000, 64, 3, 9000], K=K, mode=mode, scale_range=(1e-3, 1.0), seed=K + 70)
    off, n, d_pad = w.layout()
    m = W.tensor_mask(w)
    wm = H.tensor_word_mask(off, n, d_pad)
    # valid worker messages: random words with zero bits past each tensor end
    signs = rng.integers(0, 2**64, (K, d_pad // 64), dtype=np.uint64)
    for o, nl in zip(off, n):
        if nl % 64:
            signs[:, o // 64 + (nl - 1) // 64] &= np.uint64((1 << (nl % 64)) - 1)
    scales = (rng.random((K, w.L)) * 0.01 + 1e-4).astype(np.float32)
    x = W.initial_x(w)
    e_srv = _rand_err(rng, 1, w, 0.003)[0]
    orc = H.OracleState(w, x0=x)
    orc.e_srv[:] = e_srv
    avg_o = np.zeros(d_pad, np.float32)
    assert orc.orc.aggregate(K, mode, signs, scales, orc.x, orc.e_srv, orc.srv_signs,
                             orc.srv_scales, avg_o) == 0
    gs = H.GpuState(w, x0=x)
    gs.e_srv.copy_(torch.from_numpy(e_srv))
    avg = torch.zeros(d_pad, dtype=torch.float32, device="cuda")
    gs.saef.saef_aggregate(gs.layout, K, mode, H.dev(signs), H.dev(scales), gs.x, gs.e_srv,
                           gs.srv_signs, gs.srv_scales, avg)
    assert gs.status() == 0
    H.assert_f32_equal(H.host(avg), avg_o, m, "mean of worker messages")
    H.assert_f32_equal(H.host(gs.x), orc.x, m, "weights")
    if mode == 1:
        H.assert_f32_equal(H.host(gs.e_srv), orc.e_srv, m, "server error")
        H.assert_words_equal(H.host(gs.srv_signs, np.uint64), orc.srv_signs, wm, "server signs")
        H.assert_f32_equal(H.host(gs.srv_scales), orc.srv_scales, np.ones(w.L, bool),
                           "server scales")


@pytest.mark.parametrize("K", [1, 2, 3, 8])
def test_step_ahead_and_error_average_parity(K):
    _case(f"step ahead / error average K={K}")
    rng = np.random.default_rng(K)
    w = W.custom(ADVERSARIAL, K=K, seed=K + 300)
    m = W.tensor_mask(w)
    x = W.initial_x(w)
    e = _rand_err(rng, K, w, 0.02)
    orc = H.OracleState(w, x0=x)
    orc.e[:] = e
    assert orc.orc.step_ahead(K, orc.x, orc.e, orc.xh) == 0
    gs = H.GpuState(w, x0=x)
    gs.e.copy_(torch.from_numpy(e))
    gs.saef.saef_step_ahead(gs.layout, K, gs.x, gs.e, gs.xh)
    H.assert_f32_equal(H.host(gs.xh), orc.xh, m, "step-ahead weights")
    assert orc.orc.error_average(K, orc.e) == 0
    gs.saef.saef_error_average(gs.layout, K, gs.e)
    H.assert_f32_equal(H.host(gs.e), orc.e, m, "averaged errors")


ROUND_CASES = {
    "flat64k": W.get("flat64k"),
    "flat64k_p1": W.get("flat64k").with_(period=1, name="flat64k_p1"),
    "flat64k_pinf": W.get("flat64k").with_(period=0, name="flat64k_pinf"),
    "flat64k_sc": W.get("flat64k").with_(mode=0, name="flat64k_sc"),
    "resnet56": W.get("resnet56"),
    "resnet56_sc": W.get("resnet56").with_(mode=0, rounds=12, name="resnet56_sc"),
    "ragged_k3": W.custom(ADVERSARIAL + [70001], K=3, period=3, rounds=7,
                          scale_range=(1e-4, 1e-1), dist="laplace_zeros", seed=999),
}


@pytest.mark.parametrize("name", list(ROUND_CASES))
def test_round_parity(name):
    """saef_round over every iteration of the workload, state compared with
    the oracle after each iteration."""
    w = ROUND_CASES[name]
    _case(f"round parity {name} K={w.K} L={w.L} d={w.d} rounds={w.rounds}")
    orc = H.OracleState(w)
    gs = H.GpuState(w)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        orc.round(t, g)
        gs.round(t, g)
        H.compare_state(gs.plain(), orc, t, name)
    assert gs.status() == 0


@pytest.mark.parametrize("K,sizes", [(3, ADVERSARIAL), (8, [4096 * 3 + 17, 64, 1, 70000])])
def test_compress_momentum_parity(K, sizes):
    _case(f"compress with momentum K={K} sizes={sizes}")
    rng = np.random.default_rng(K + 17)
    w = W.custom(sizes, K=K, scale_range=(1e-3, 1.0), seed=K + 77)
    off, n, d_pad = w.layout()
    msk = W.tensor_mask(w)
    g = W.gradients(w, 0)
    e = _rand_err(rng, K, w)
    m0 = _rand_err(rng, K, w, 0.5)
    mu = np.float32(0.9)
    orc = H.OracleState(w, mu=0.9)
    orc.e[:] = e
    orc.m[:] = m0
    assert orc.orc.compress_momentum(K, LR, mu, g, orc.m, orc.e, orc.signs, orc.scales) == 0
    gs = H.GpuState(w, mu=0.9)
    gs.e.copy_(torch.from_numpy(e))
    gs.m.copy_(torch.from_numpy(m0))
    gs.saef.saef_compress_momentum(gs.layout, K, float(LR), float(mu), H.dev(g), gs.m, gs.e,
                                   gs.signs, gs.scales)
    assert gs.status() == 0
    H.assert_words_equal(H.host(gs.signs, np.uint64), orc.signs,
                         H.tensor_word_mask(off, n, d_pad), "signs")
    H.assert_f32_equal(H.host(gs.scales), orc.scales, np.ones(w.L, bool), "scales")
    H.assert_f32_equal(H.host(gs.e), orc.e, msk, "errors")
    H.assert_f32_equal(H.host(gs.m), orc.m, msk, "momentum buffers")


MOMENTUM_CASES = {
    "flat64k": W.get("flat64k"),
    "resnet56": W.get("resnet56").with_(rounds=12),
    "ragged_sc": W.custom(ADVERSARIAL + [70001], K=3, period=3, rounds=7, mode=0,
                          scale_range=(1e-4, 1e-1), dist="laplace_zeros", seed=998),
}


@pytest.mark.parametrize("name", list(MOMENTUM_CASES))
def test_round_momentum_parity(name):
    """saef_round_momentum (mu = 0.9, the paper's momentum constant) over
    every iteration, state and momentum buffers compared with the oracle."""
    w = MOMENTUM_CASES[name]
    _case(f"momentum round parity {name} K={w.K} L={w.L} rounds={w.rounds}")
    orc = H.OracleState(w, mu=0.9)
    gs = H.GpuState(w, mu=0.9)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        orc.round(t, g)
        gs.round(t, g)
        H.compare_state(gs.plain(), orc, t, name)
    assert gs.status() == 0


def test_round_momentum_zero_equals_round():
    """mu = 0 with zero momentum buffers is the plain iteration, bit for bit."""
    w = W.get("resnet56").with_(period=3, rounds=5)
    _case("momentum 0 vs plain round")
    a = H.GpuState(w)
    b = H.GpuState(w, mu=0.0)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        a.round(t, g)
        b.round(t, g)
    pa, pb = a.plain(), b.plain()
    for key in pa:
        assert pa[key].tobytes() == pb[key].tobytes(), key


def test_round_equals_eager_ops():
    """The fused iteration and the four separate entry points called in
    Algorithm 1 order give identical states."""
    w = W.get("resnet56").with_(period=3, rounds=7)
    _case("fused round vs eager ops, resnet56 period 3")
    fused = H.GpuState(w)
    eager = H.GpuState(w)
    S = eager.saef
    for t in range(w.rounds):
        g = W.gradients(w, t)
        fused.round(t, g)
        eager.g.copy_(torch.from_numpy(g))
        if (t + 1) % w.period == 0:
            S.saef_error_average(eager.layout, w.K, eager.e)
        S.saef_step_ahead(eager.layout, w.K, eager.x, eager.e, eager.xh)
        S.saef_compress(eager.layout, w.K, w.lr, eager.g, eager.e, eager.signs, eager.scales)
        S.saef_aggregate(eager.layout, w.K, w.mode, eager.signs, eager.scales, eager.x,
                         eager.e_srv, eager.srv_signs, eager.srv_scales)
        a = fused.plain()
        torch.cuda.synchronize()
        m = W.tensor_mask(w)
        for key, tens in (("e", eager.e), ("e_srv", eager.e_srv), ("x", eager.x),
                          ("xh", eager.xh)):
            H.assert_f32_equal(a[key], H.host(tens), m, f"t={t} {key}")
        for key, tens in (("scales", eager.scales), ("srv_scales", eager.srv_scales)):
            H.assert_f32_equal(a[key], H.host(tens), np.ones(w.L, bool), f"t={t} {key}")
        assert np.array_equal(a["signs"], H.host(eager.signs, np.uint64)), t
        assert np.array_equal(a["srv_signs"], H.host(eager.srv_signs, np.uint64)), t


def test_repeat_runs_are_bit_identical():
    w = W.get("resnet56").with_(rounds=4)
    _case("determinism resnet56 x2")
    outs = []
    for _ in range(2):
        gs = H.GpuState(w)
        for t in range(w.rounds):
            gs.round(t, W.gradients(w, t))
        outs.append(gs.plain())
    for key in outs[0]:
        assert outs[0][key].tobytes() == outs[1][key].tobytes(), key


def test_out_of_range_sets_status_and_clears():
    w = W.custom([1000, 64], K=2, seed=5)
    _case("range error flag")
    gs = H.GpuState(w)
    g = W.gradients(w, 0)
    g[1, 17] = 1e7                      # lr * g = 1e6 >= 2^19
    gs.round(0, g)
    assert gs.status() == gs.saef.ERANGE
    assert gs.status() == 0             # the flag is cleared by the read
    g = W.gradients(w, 1)
    g[0, 3] = np.inf
    gs.saef.saef_compress(gs.layout, 2, 0.1, H.dev(g), gs.e, gs.signs, gs.scales)
    assert gs.status() == gs.saef.ERANGE


def test_invalid_arguments_are_rejected():
    w = W.custom([100], K=2, seed=5)
    _case("invalid arguments")
    gs = H.GpuState(w)
    S = gs.saef
    with pytest.raises(S.SaefError) as ex:       # K above the layout's k_max
        S.saef_step_ahead(gs.layout, 3, gs.x, gs.e, gs.xh)
    assert ex.value.rc == S.EINVAL
    with pytest.raises(S.SaefError):             # xh overlaps e
        S.saef_step_ahead(gs.layout, 2, gs.x, gs.e, gs.e)
    with pytest.raises(S.SaefError):             # mode out of range
        S.saef_aggregate(gs.layout, 2, 5, gs.signs, gs.scales, gs.x)
    with pytest.raises(S.SaefError):             # double-way needs the server buffers
        S.saef_aggregate(gs.layout, 2, 1, gs.signs, gs.scales, gs.x)
    with pytest.raises(S.SaefError):             # g and e overlap
        S.saef_compress(gs.layout, 2, 0.1, gs.e, gs.e, gs.signs, gs.scales)


def test_profile_sampling():
    """saef_profile_enable with every = 3 stamps dispatches 0, 3, 6 of each
    timed kind and nothing else; every < 1 is rejected; the iterations give
    the same bits as unprofiled ones."""
    w = W.custom([5000, 70, 4097], K=2, period=0, seed=6)
    _case("profile sampling")
    gs, ref = H.GpuState(w), H.GpuState(w)
    S = gs.saef
    with pytest.raises(S.SaefError) as ex:
        S.saef_profile_enable(gs.layout, 4, kinds=("compress",), every=0)
    assert ex.value.rc == S.EINVAL
    S.saef_profile_enable(gs.layout, 10, kinds=("compress", "aggregate"), every=3)
    for t in range(7):
        g = W.gradients(w, t)
        gs.round(t, g)
        ref.round(t, g)
    prof = S.saef_profile_read(gs.layout)
    S.saef_profile_enable(gs.layout, 0)
    assert prof["compress"][0] == 3 and prof["aggregate"][0] == 3, prof
    assert prof["compress"][1] > 0.0 and prof["aggregate"][1] > 0.0, prof
    assert all(c == 0 for k, (c, _) in prof.items() if k not in ("compress", "aggregate")), prof
    for name in ("x", "e", "e_srv", "signs", "scales"):
        assert torch.equal(getattr(gs, name), getattr(ref, name)), name


# ---------------------------------------------------------------- two halves, EF, mismatch

SPLIT_CASES = {
    "resnet56_dc": W.get("resnet56").with_(period=4, rounds=9),
    "ragged_sc": W.custom(ADVERSARIAL + [70001], K=3, period=3, rounds=7, mode=0,
                          scale_range=(1e-4, 1e-1), dist="laplace_zeros", seed=998),
    "flat64k_no_avg": W.get("flat64k").with_(period=0, rounds=6),
    # the mismatch kernel keeps up to 4, 8 or 16 workers in registers, and
    # reads the errors twice above 16
    "k12_avg": W.custom(ADVERSARIAL + [9000], K=12, period=3, rounds=4, seed=41),
    "k20_dc": W.custom([4097, 65, 30000], K=20, period=2, rounds=4, seed=42),
}


@pytest.mark.parametrize("variant", [0, 1], ids=["ef", "saef"])
@pytest.mark.parametrize("name", list(SPLIT_CASES))
def test_round_halves_parity(name, variant):
    """saef_round_begin (with the mismatch bounds) + saef_round_end against
    the oracle's two halves, every iteration; EF writes one row of xh."""
    w = SPLIT_CASES[name]
    _case(f"round halves {name} variant={variant} K={w.K} L={w.L} rounds={w.rounds}")
    orc = H.OracleState(w)
    gs = H.GpuState(w)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        want = orc.begin(t, variant)
        got = gs.begin(t, variant)
        H.assert_mismatch_close(got, want, w, w.K, f"{name} t={t}")
        orc.end(t, g)
        gs.end(t, g)
        H.compare_state(gs.plain(), orc, t, name)
    assert gs.status() == 0


def test_round_halves_equal_round():
    """begin(SAEF) + end is saef_round, bit for bit (pending form included)."""
    w = W.get("resnet56").with_(period=3, rounds=6)
    _case("round halves vs saef_round")
    a = H.GpuState(w)
    b = H.GpuState(w)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        a.round(t, g)
        b.begin(t, 1, mismatch=(t % 2 == 0))
        b.end(t, g)
    torch.cuda.synchronize()
    for key in ("e", "e_srv", "x", "xh", "signs", "scales", "srv_signs", "srv_scales"):
        assert torch.equal(getattr(a, key), getattr(b, key)), key


@pytest.mark.parametrize("variant", [0, 1], ids=["ef", "saef"])
def test_closed_loop_quadratic(variant):
    """Gradients that depend on the evaluation point: a noisy quadratic,
    g^(k) = (xh - x*) / 2 + noise^(k), computed with fp32 elementwise torch
    ops between the two halves on the GPU and with numpy on the host (the
    same correctly rounded operations).  The two branches now follow
    different trajectories, and each matches the oracle bit for bit."""
    w = W.get("resnet56").with_(period=0, rounds=8)
    _case(f"closed-loop quadratic variant={variant}")
    off, n, d_pad = w.layout()
    rng = np.random.default_rng(2024)
    xstar = (rng.standard_normal(d_pad) * 0.05).astype(np.float32)
    orc = H.OracleState(w)
    gs = H.GpuState(w)
    xstar_d = torch.from_numpy(xstar).cuda()
    for t in range(w.rounds):
        noise = (rng.standard_normal((w.K, d_pad)) * 0.01).astype(np.float32)
        want = orc.begin(t, variant)
        got = gs.begin(t, variant)
        H.assert_mismatch_close(got, want, w, w.K, f"closed loop t={t}")
        rows = orc.xh if variant == 1 else np.repeat(orc.xh[:1], w.K, axis=0)
        g_host = (np.float32(0.5) * (rows - xstar)).astype(np.float32) + noise
        xh_d = gs.xh if variant == 1 else gs.xh[:1].expand(w.K, d_pad)
        g_dev = (0.5 * (xh_d - xstar_d)) + torch.from_numpy(noise).cuda()
        orc.end(t, g_host)
        gs.end(t, g_dev.contiguous())
        H.compare_state(gs.plain(), orc, t, f"closed loop v{variant}")
    assert gs.status() == 0


def test_round_halves_invalid():
    w = W.custom([100], K=2)
    gs = H.GpuState(w)
    s = gs.saef
    with pytest.raises(s.SaefError):  # unknown variant
        s.saef_round_begin(gs.layout, 0, 0, 2, 1, 2, gs.e, gs.e_srv, gs.x, gs.xh, gs.signs,
                           gs.scales, gs.srv_signs, gs.srv_scales)
    with pytest.raises(s.SaefError):  # EF evaluation point aliases the weights
        s.saef_round_begin(gs.layout, 0, 0, 2, 1, 0, gs.e, gs.e_srv, gs.x, gs.x, gs.signs,
                           gs.scales, gs.srv_signs, gs.srv_scales)
    with pytest.raises(s.SaefError):  # mu without a momentum buffer
        s.saef_round_end(gs.layout, 0, 0, 2, 0.1, 0.9, 1, gs.g, None, gs.e, gs.e_srv, gs.x,
                         gs.signs, gs.scales, gs.srv_signs, gs.srv_scales)
    with pytest.raises(s.SaefError):  # mismatch bounds need the server error in DC
        s.saef_round_begin(gs.layout, 0, 0, 2, 1, 1, gs.e, None, gs.x, gs.xh, gs.signs,
                           gs.scales, gs.srv_signs, gs.srv_scales,
                           torch.zeros(2, dtype=torch.float64, device="cuda"))
    torch.cuda.synchronize()
    assert gs.status() == 0


# ---------------------------------------------------------------- HIP graphs

def test_graph_replay_parity():
    """saef_round captured in HIP graphs (torch.cuda.CUDAGraph, the library
    launching on the capture stream): one graph per kind of iteration (t = 0
    with plain state, pending state, pending state with error averaging),
    replayed over the iterations with the gradients copied in eagerly between
    replays and the state checked against the oracle after every replay."""
    w = W.get("resnet56").with_(period=4, rounds=10)
    _case(f"graph replay resnet56 K={w.K} rounds={w.rounds}")
    orc = H.OracleState(w)
    gs = H.GpuState(w)
    S = gs.saef
    graphs = {}
    for t in range(w.rounds):
        kind = (t > 0, (t + 1) % w.period == 0)
        if kind not in graphs:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                S.saef_round(gs.layout, t, w.period, gs.K, w.lr, w.mode, gs.g, gs.e, gs.e_srv,
                             gs.x, gs.xh, gs.signs, gs.scales, gs.srv_signs, gs.srv_scales)
            graphs[kind] = graph
        grad = W.gradients(w, t)
        gs.g.copy_(torch.from_numpy(grad))
        graphs[kind].replay()
        torch.cuda.synchronize()
        orc.round(t, grad)
        H.compare_state(gs.plain(), orc, t, "graph replay")
    assert len(graphs) == 3
    assert gs.status() == 0
