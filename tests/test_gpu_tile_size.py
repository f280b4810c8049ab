"""The results do not depend on the work-tile size.

The per-tensor L1 norm is an exact integer sum, so the scales, and with them
every sign word, error and weight, are independent of how the tensors are cut
into tiles and of the order in which tiles are reduced.  The sign path built
with 4096-element tiles (other tile counts, grids, XCD run orders and exact
sums flushed across two passes per lane) must give byte-identical state to
the default 2048-element build after every iteration: resnet56 (167 tensors,
20 iterations with averaging), a ragged double-way layout and a single-way
layout with momentum.  Each build runs in a fresh process of its own
(SAEF_LIBRARY selects the library)."""
import os
import subprocess
import sys

import numpy as np
import pytest

from paper_2008_05823_amd import build as B

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(lib: str, out: str):
    env = dict(os.environ, SAEF_LIBRARY=lib)
    print(f"[tile-size] running {os.path.basename(lib)}", flush=True)
    subprocess.run([sys.executable, "-m", "tests.tile_size_child", out], cwd=ROOT, env=env,
                   check=True, timeout=600)


@pytest.mark.timeout(900)
def test_tile_size_does_not_change_any_byte(tmp_path):
    if not os.path.exists(B.LIB_TILE_VARIANT):
        pytest.fail(f"{B.LIB_TILE_VARIANT} is missing: run __graft_entry__.build()")
    a, b = tmp_path / "t2048.npz", tmp_path / "t4096.npz"
    _run(B.LIB, str(a))
    _run(B.LIB_TILE_VARIANT, str(b))
    ra, rb = np.load(a), np.load(b)
    assert sorted(ra.files) == sorted(rb.files)
    tiles = {k: (int(ra[k]), int(rb[k])) for k in ra.files if k.endswith(".n_tiles")}
    for k, (na, nb) in tiles.items():
        assert na > nb, (k, na, nb)  # the variant really cuts the tensors differently
    differ = [k for k in ra.files if not k.endswith(".n_tiles")
              and not np.array_equal(ra[k].view(np.uint8), rb[k].view(np.uint8))]
    assert not differ, f"{len(differ)} arrays differ between tile sizes, first: {differ[:5]}"
