"""The piecewise, threaded oracle used by the full-size parity tests equals
the oracle's whole-layout iteration bit for bit (CPU only)."""
import numpy as np
import pytest

from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H
from tests.split_oracle import SplitOracle, rows_equal

CASES = [
    # sizes, K, period, mode, dist
    ([4097, 64, 3, 1000, 130, 1], 3, 2, 1, "normal"),
    ([65, 127, 2049, 700], 5, 0, 1, "laplace_zeros"),
    ([300, 5000, 1, 64], 4, 3, 0, "normal_outliers"),
    ([20000], 8, 2, 1, "normal"),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_split_oracle_equals_whole_layout(case):
    sizes, K, period, mode, dist = CASES[case]
    w = W.custom(sizes, K=K, period=period, rounds=5, dist=dist, mode=mode,
                 scale_range=(1e-3, 1e-1), seed=W.SEED_BASE + 300 + case)
    ref = H.OracleState(w)
    # small chunks: the first half runs on pieces of tensors
    so = SplitOracle(w, threads=4, chunk=128)
    for t in range(w.rounds):
        g = W.gradients(w, t)
        ref.round(t, g)
        so.round(t, g)
        for name in ("e", "e_srv", "x", "xh", "signs", "srv_signs"):
            a, b = getattr(so, name), getattr(ref, name)
            assert rows_equal(a, b, threads=3), (case, t, name)
        assert np.array_equal(so.scales.view(np.uint32), ref.scales.view(np.uint32)), (case, t)
        if mode == 1:
            assert np.array_equal(so.srv_scales.view(np.uint32),
                                  ref.srv_scales.view(np.uint32)), (case, t)


def test_rows_equal_finds_a_single_flipped_bit():
    rng = np.random.default_rng(3)
    a = rng.standard_normal((3, 5000)).astype(np.float32)
    b = a.copy()
    assert rows_equal(a, b, threads=4)
    b.view(np.uint32)[2, 4999] ^= 1
    assert not rows_equal(a, b, threads=4)
    c = a.copy()
    c[0, 0] = -0.0 if a[0, 0] == 0 else a[0, 0]
    c.view(np.uint32)[0, 0] ^= 0x80000000  # sign of the first value
    assert not rows_equal(a, c, threads=4)
