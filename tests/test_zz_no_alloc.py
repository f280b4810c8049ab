"""saef_round_noalloc (the allocation-free iteration: tile partial sums in
the library's static device scratch) gives the same state as saef_round, bit
for bit, on two calls in a row of which the second has a smaller layout, and
refuses a layout whose partial sums do not fit the scratch."""
import numpy as np
import pytest
import torch

from paper_2008_05823_amd import saef
from paper_2008_05823_amd import workloads as W
from tests import gpu_harness as H

pytestmark = pytest.mark.gpu


def _state(w, x0):
    off, n, d_pad = w.layout()
    f32 = dict(dtype=torch.float32, device="cuda")
    i64 = dict(dtype=torch.int64, device="cuda")
    return dict(x=torch.from_numpy(x0.copy()).cuda(), e=torch.zeros((w.K, d_pad), **f32),
                e_srv=torch.zeros(d_pad, **f32), xh=torch.zeros((w.K, d_pad), **f32),
                signs=torch.zeros((w.K, d_pad // 64), **i64), scales=torch.zeros((w.K, w.L), **f32),
                srv_signs=torch.zeros(d_pad // 64, **i64), srv_scales=torch.zeros(w.L, **f32))


def _run(fn, lay, w, st, t, g, mode):
    fn(lay, t, w.period, w.K, w.lr, mode, g, st["e"], st["e_srv"], st["x"], st["xh"], st["signs"],
       st["scales"], st["srv_signs"], st["srv_scales"])


def _assert_same(a, b, tag):
    for k in a:
        x, y = a[k].cpu().numpy(), b[k].cpu().numpy()
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), f"{tag}: {k} differs"


# a 3145-tile layout (K = 8), then a smaller one (K = 3, single-way in one case)
CASES = [
    (dict(sizes=None, K=8, period=2, mode=1), dict(sizes=[5000, 70, 64, 1], K=3, period=0, mode=1)),
    (dict(sizes=[300000, 4097, 65], K=5, period=3, mode=1), dict(sizes=[129, 2048], K=2, period=2,
                                                                   mode=0)),
]


def _workload(spec, seed):
    if spec["sizes"] is None:
        rng = np.random.default_rng(2048)
        sizes = np.concatenate([rng.integers(1, 300001, 40), rng.integers(1, 200, 6), [1, 64]])
        spec = dict(spec, sizes=sizes.tolist())
    return W.custom(spec["sizes"], K=spec["K"], period=spec["period"], rounds=3,
                    dist="laplace_zeros", scale_range=(1e-4, 1e-1), seed=seed, mode=spec["mode"])


@pytest.mark.parametrize("case", range(len(CASES)))
def test_noalloc_round_equals_round(case):
    for i, spec in enumerate(CASES[case]):
        w = _workload(spec, W.SEED_BASE + 700 + 10 * case + i)
        off, n, d_pad = w.layout()
        x0 = W.initial_x(w)
        lay = saef.Layout(off, n, d_pad, w.K)
        ref, got = _state(w, x0), _state(w, x0)
        for t in range(w.rounds):  # t = 0 plain, then pending corrections, averaging when due
            g = torch.from_numpy(W.gradients(w, t)).cuda()
            _run(saef.saef_round, lay, w, ref, t, g, w.mode)
            _run(saef.saef_round_noalloc, lay, w, got, t, g, w.mode)
            torch.cuda.synchronize()
            _assert_same(ref, got, f"case {case} call {i} t={t}")
        assert saef.saef_status(lay) == saef.OK
        # the plain state agrees with the oracle too
        orc = H.OracleState(w, x0=x0)
        for t in range(w.rounds):
            orc.round(t, W.gradients(w, t))
        gs = H.GpuState(w, x0=x0)
        gs.layout.close()
        gs.layout = lay
        for k in ("x", "e", "e_srv", "xh", "signs", "scales", "srv_signs", "srv_scales"):
            setattr(gs, k, got[k])
        H.compare_state(gs.plain(), orc, w.rounds - 1, f"noalloc case {case} call {i}")
        lay.close()


def test_noalloc_refuses_layouts_beyond_the_scratch():
    """One 2^28-element tensor is 131072 tiles: K = 8 needs 9 rows of tile
    sums (18 MiB) and runs; K = 15 needs 16 rows (32 MiB) plus the second
    level, more than the 32 MiB scratch: SAEF_EINVAL, while saef_round (the
    layout's own scratch) runs the same call."""
    n = 1 << 28
    lay = saef.Layout([0], [n], n, 16)
    f32 = dict(dtype=torch.float32, device="cuda")
    for K, fits in ((8, True), (15, False)):
        st = dict(x=torch.zeros(n, **f32), e=torch.zeros((K, n), **f32),
                  e_srv=torch.zeros(n, **f32), xh=torch.zeros((K, n), **f32),
                  signs=torch.zeros((K, n // 64), dtype=torch.int64, device="cuda"),
                  scales=torch.zeros((K, 1), **f32),
                  srv_signs=torch.zeros(n // 64, dtype=torch.int64, device="cuda"),
                  srv_scales=torch.zeros(1, **f32))
        g = torch.zeros((K, n), **f32)
        w = W.custom([n], K=K, period=0)
        _run(saef.saef_round, lay, w, st, 0, g, 1)
        if fits:
            _run(saef.saef_round_noalloc, lay, w, st, 1, g, 1)
        else:
            with pytest.raises(saef.SaefError) as err:
                _run(saef.saef_round_noalloc, lay, w, st, 1, g, 1)
            assert err.value.rc == saef.EINVAL
        torch.cuda.synchronize()
        del st, g
        torch.cuda.empty_cache()
    assert saef.saef_status(lay) == saef.OK
    lay.close()
