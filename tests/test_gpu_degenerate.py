"""Degenerate cases of the method on the GPU, against the oracle, bit for bit
(needs an MI355X).

- all-zero gradients: sign(0) = +1 gives scale 0 and no error; with Top-K
  every key is equal, so the whole tensor is one tie group cut by index (the
  candidate path at its worst case: every element is a candidate);
- one worker (K = 1), and averaging in every iteration (p = 1);
- many tiny tensors (n = 1 .. 100);
- crafted values: signed zeros, subnormals, magnitudes just below the
  exact-sum limit 2^19 of the scaled sign.
"""
import numpy as np
import pytest

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H
from tests.test_gpu_topk import TopkGpu, TopkOracle, compare_topk

pytestmark = pytest.mark.gpu


def _case(msg):
    print(f"[case] {msg}", flush=True)


def _crafted(rng, shape):
    """Signed zeros, subnormals, tiny and large magnitudes (|v| < 2^19 / 4,
    so that e + lr g stays inside the exact-sum range)."""
    v = rng.standard_normal(shape).astype(np.float32)
    v *= np.float32(2.0) ** rng.integers(-40, 16, shape).astype(np.float32)
    pick = rng.random(shape)
    v[pick < 0.05] = 0.0
    v[(pick >= 0.05) & (pick < 0.10)] = -0.0
    sub = (pick >= 0.10) & (pick < 0.15)
    v[sub] = (np.float32(1e-40) * rng.standard_normal(int(sub.sum()))).astype(np.float32)
    big = (pick >= 0.15) & (pick < 0.17)
    v[big] = np.float32(131000.0) * np.sign(rng.standard_normal(int(big.sum()))).astype(np.float32)
    return v


CASES = {
    "zeros_k4": (W.custom([5000, 64, 1, 70001], K=4, period=3, rounds=4, seed=1), "zeros"),
    "single_worker": (W.custom([4097, 3, 1000], K=1, period=2, rounds=5, seed=2), "grad"),
    "average_every_iteration": (W.custom([300, 65, 8193], K=3, period=1, rounds=4, seed=3), "grad"),
    "many_tiny_tensors": (W.custom([1 + (i * 37) % 100 for i in range(300)], K=2, period=4,
                                   rounds=5, seed=4), "grad"),
    "crafted_values": (W.custom([4096, 77, 20000], K=3, period=0, rounds=4, seed=5), "crafted"),
}


def _grads(w, t, src):
    off, n, d_pad = w.layout()
    if src == "zeros":
        return np.zeros((w.K, d_pad), np.float32)
    if src == "crafted":
        g = _crafted(np.random.default_rng(100 + t), (w.K, d_pad))
        g[:, ~W.tensor_mask(w)] = 0.0
        return g
    return W.gradients(w, t)


@pytest.mark.parametrize("name", list(CASES))
def test_degenerate_sign(name):
    w, src = CASES[name]
    _case(f"degenerate scaled sign {name}")
    orc = H.OracleState(w)
    gs = H.GpuState(w)
    for t in range(w.rounds):
        g = _grads(w, t, src)
        orc.round(t, g)
        gs.round(t, g)
        H.compare_state(gs.plain(), orc, t, name)
    assert gs.status() == 0


@pytest.mark.parametrize("pct", [1, 50], ids=["1pct", "50pct"])
@pytest.mark.parametrize("name", list(CASES))
def test_degenerate_topk(name, pct):
    w, src = CASES[name]
    keep = W.topk_keep(w, pct)
    _case(f"degenerate top-k {name} {pct}%")
    orc = TopkOracle(w, keep)
    gs = TopkGpu(w, keep)
    for t in range(w.rounds):
        g = _grads(w, t, src)
        orc.round(t, g)
        gs.round(t, g)
        compare_topk(gs, orc, t, f"{name} {pct}%", mode=w.mode)
    assert gs.status() == 0
