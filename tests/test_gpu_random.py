"""Randomized parity of the HIP library with the CPU oracle (needs an
MI355X): seeded random tensor lists (1 to 24 tensors of 1 to 200,000
elements), worker counts, modes, averaging periods, gradient distributions,
momentum, the EF or SAEF branch, and for Top-K random kept percentages.
Every case is fixed by its seed, so a failure names a reproducible case.
"""
import math

import numpy as np
import pytest

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H
from tests.test_gpu_topk import TopkGpu, TopkOracle, compare_topk

pytestmark = pytest.mark.gpu

DISTS = ("normal", "laplace_zeros", "normal_outliers")


def _case(msg):
    print(f"[case] {msg}", flush=True)


def _random_workload(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 25))
    sizes = [int(math.exp(rng.uniform(0.0, math.log(200_000)))) for _ in range(L)]
    K = int(rng.integers(1, 21))
    return W.custom(sizes, K=K, period=int(rng.choice([0, 1, 2, 3, 5])),
                    rounds=int(rng.integers(3, 5)), dist=str(rng.choice(DISTS)),
                    seed=seed, mode=int(rng.integers(0, 2)),
                    scale_range=(1e-4, float(rng.choice([1e-2, 1.0])))), rng


@pytest.mark.parametrize("seed", range(1000, 1032))
def test_random_sign_parity(seed):
    w, rng = _random_workload(seed)
    mu = 0.9 if rng.random() < 0.3 else None
    halves = rng.random() < 0.4
    variant = int(rng.integers(0, 2)) if halves else 1
    _case(f"random scaled sign seed={seed} L={w.L} d={w.d} K={w.K} mode={w.mode} "
          f"period={w.period} dist={w.dist} mu={mu} halves={halves} variant={variant}")
    orc = H.OracleState(w, mu=mu)
    gs = H.GpuState(w, mu=mu)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        if halves:
            want = orc.begin(t, variant)
            got = gs.begin(t, variant)
            H.assert_mismatch_close(got, want, w, w.K, f"seed {seed} t={t}")
            orc.end(t, g)
            gs.end(t, g)
        else:
            orc.round(t, g)
            gs.round(t, g)
        H.compare_state(gs.plain(), orc, t, f"seed {seed}")
    assert gs.status() == 0


@pytest.mark.parametrize("seed", range(2000, 2024))
def test_random_topk_parity(seed):
    w, rng = _random_workload(seed)
    pct = float(rng.choice([0.5, 1.0, 10.0, 50.0, 100.0]))
    mu = 0.9 if rng.random() < 0.3 else None
    keep = W.topk_keep(w, pct)
    _case(f"random top-k seed={seed} L={w.L} d={w.d} K={w.K} mode={w.mode} "
          f"period={w.period} dist={w.dist} pct={pct} mu={mu}")
    orc = TopkOracle(w, keep, mu=mu)
    gs = TopkGpu(w, keep, mu=mu)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        orc.round(t, g)
        gs.round(t, g)
        compare_topk(gs, orc, t, f"seed {seed}", mode=w.mode)
    assert gs.status() == 0
