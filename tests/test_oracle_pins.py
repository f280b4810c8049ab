"""The CPU oracle against the paper and the mathematics (no GPU needed)."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import exact, oracle_pins as P


@pytest.fixture(scope="module")
def libpath():
    O.lib()
    return O.LIB


@pytest.mark.parametrize("pin", P.QUICK_PINS, ids=lambda f: f.__name__)
def test_pin(libpath, pin):
    pin(libpath)


def test_l1_fixed_equals_exact_integer_sum():
    """The exact L1 sum equals the Python big-integer sum of floor(|v| 2^80),
    and its binary64 rounding equals math.fsum of the truncated terms."""
    import math
    rng = np.random.default_rng(11)
    for trial in range(20):
        v = P._rand_values(rng, int(rng.integers(1, 3000)))
        if trial == 0:
            v[:3] = [np.float32(524287.97), -np.float32(2.0 ** -80), np.float32(1.5 * 2 ** -80)]
        rc, S = O.l1_fixed(v)
        assert rc == O.OK
        assert S == exact.exact_l1_fixed(v)
        terms = [exact.exact_l1_fixed([x]) * 2.0 ** -80 for x in v.tolist()]
        assert float(S) * 2.0 ** -80 == math.fsum(terms)


def test_sign_of_zero_is_plus_one(libpath):
    off, n, d_pad = P._one_tensor_layout([3])
    orc = O.Oracle(off, n, d_pad, libpath)
    g = np.array([[0.0, -0.0, -1e-30] + [0.0] * 61], np.float32)
    e = np.zeros_like(g)
    signs = np.zeros((1, 1), np.uint64)
    scales = np.zeros((1, 1), np.float32)
    assert orc.compress(1, np.float32(1.0), g, e, signs, scales) == O.OK
    assert int(signs[0, 0]) == 0b011


@pytest.mark.parametrize("bad", [np.float32(524288.0), np.float32(-6e5), np.float32(np.inf),
                                 np.float32(np.nan)])
def test_out_of_range_value_is_reported(libpath, bad):
    off, n, d_pad = P._one_tensor_layout([10])
    orc = O.Oracle(off, n, d_pad, libpath)
    g = np.zeros((2, d_pad), np.float32)
    g[1, 4] = bad / np.float32(0.1) if np.isfinite(bad) else bad
    e = np.zeros_like(g)
    signs = np.zeros((2, 1), np.uint64)
    scales = np.zeros((2, 1), np.float32)
    assert orc.compress(2, np.float32(0.1), g, e, signs, scales) == O.ERANGE


@pytest.mark.parametrize("off,n,d_pad", [
    ([32], [10], 64),            # offset not a multiple of 64
    ([0, 64], [100, 10], 192),   # overlap
    ([0], [0], 64),              # empty tensor
    ([0], [65], 64),             # past d_pad
])
def test_invalid_layout_is_rejected(libpath, off, n, d_pad):
    orc = O.Oracle(np.array(off), np.array(n), d_pad, libpath)
    K = 1
    g = np.zeros((K, d_pad), np.float32)
    e = np.zeros_like(g)
    signs = np.zeros((K, max(1, d_pad // 64)), np.uint64)
    scales = np.zeros((K, len(off)), np.float32)
    assert orc.compress(K, np.float32(0.1), g, e, signs, scales) == O.EINVAL


def test_zero_workers_rejected(libpath):
    off, n, d_pad = P._one_tensor_layout([10])
    orc = O.Oracle(off, n, d_pad, libpath)
    x = np.zeros(d_pad, np.float32)
    e = np.zeros((1, d_pad), np.float32)
    assert orc.step_ahead(0, x, e, e.copy()) == O.EINVAL
