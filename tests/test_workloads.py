"""The synthetic workloads have the shapes of the models they stand for."""
import os

import numpy as np
import pytest

from paper_2008_05823_amd import workloads as W


@pytest.mark.parametrize("name,L,d,K,largest", [
    ("flat64k", 1, 65536, 4, 65536),
    ("resnet56", 167, 853018, 8, 36864),
    ("resnet50", 161, 25557032, 8, 2359296),
    ("bert_base", 199, 109482240, 16, 30522 * 768),
    ("flat256m", 1, 1 << 28, 8, 1 << 28),
])
def test_shapes(name, L, d, K, largest):
    w = W.get(name)
    off, n, d_pad = w.layout()
    assert w.L == L and w.d == d and w.K == K and n.max() == largest
    assert (off % 64 == 0).all() and d_pad % 64 == 0
    assert (off[1:] >= off[:-1] + n[:-1]).all() and off[-1] + n[-1] <= d_pad


def test_gradients_are_seeded_and_independent_per_round_and_worker():
    w = W.custom([1000, 77], K=3, seed=4)
    a = W.gradients(w, 0)
    assert np.array_equal(a, W.gradients(w, 0))
    assert not np.array_equal(a[0], a[1])
    assert not np.array_equal(a, W.gradients(w, 1))
    assert (a[:, ~W.tensor_mask(w)] == 0).all()


def test_distributions():
    w = W.custom([200000], K=1, dist="laplace_zeros", scale_range=(1e-3, 1e-3), seed=1)
    g = W.gradient(w, 0, 0)
    assert abs((g == 0).mean() - 0.05) < 0.005
    nz = g[g != 0].astype(np.float64)
    assert abs(np.abs(nz).mean() - 1e-3) < 2e-5          # Laplace(0, b): E|g| = b
    w = W.custom([200000], K=1, dist="normal_outliers", scale_range=(1e-2, 1e-2), seed=1)
    g = W.gradient(w, 0, 0)
    out = np.isclose(np.abs(g), 1.0)                       # +-100 sigma
    assert abs(out.mean() - 0.01) < 0.002
    assert abs(g[~out].std() - 1e-2) < 2e-4


def test_per_tensor_scales_log_uniform():
    s = W.tensor_scales(W.get("resnet50"))
    assert s.min() >= 1e-5 and s.max() <= 1e-2 and len(s) == 161


def test_byte_model():
    assert W.algorithmic_bytes_per_param(8) == 182.125
    assert W.algorithmic_bytes_per_param(4) == 101.125
    assert W.algorithmic_bytes_per_param(16) == 344.125
    assert W.algorithmic_bytes_per_param(8, mode=0) == 12 + 20.25 * 8


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU: --gpus N > 1 exits with a message (no GPU
    is touched before the check)."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    res = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr


def test_topk_keep_and_byte_models():
    from paper_2008_05823_amd import workloads as W
    w = W.custom([1, 99, 100, 101, 12345], K=2)
    assert W.topk_keep(w, 1).tolist() == [1, 1, 1, 2, 124]
    assert W.topk_keep(w, 100).tolist() == [1, 99, 100, 101, 12345]
    assert W.topk_keep(w, 5).tolist() == [1, 5, 5, 6, 618]
    # sign path, K = 8, double-way: 20.125 + 20.25 K
    assert W.algorithmic_bytes_per_param(8) == 20.125 + 20.25 * 8
    assert W.algorithmic_bytes_per_param(8, averaging=True) == 20.125 + 20.25 * 8 + 32
    assert W.algorithmic_bytes_per_param(8, momentum=True) == 20.125 + 28.25 * 8
    tk = W.topk_algorithmic_bytes_per_param(8, 0.01)
    assert abs(tk["worker"] - 8 * (12 + 3 / 16 + 0.04)) < 1e-12
