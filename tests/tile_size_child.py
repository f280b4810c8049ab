"""Child process of the tile-size determinism test (GPU): runs sign-path
iterations through whichever library SAEF_LIBRARY names and writes, per
iteration, a SHA-256 of every state array's bytes (and the final arrays)
to an .npz file.  Usage: python -m tests.tile_size_child OUT.npz"""
import hashlib
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def cases():
    from paper_2008_05823_amd import workloads as W
    yield "resnet56", W.get("resnet56"), None, 1
    yield "ragged_dc", W.custom([70000, 4095, 4097, 12289, 1, 300000, 63, 8192], K=5, period=3,
                                rounds=6, dist="laplace_zeros", scale_range=(1e-4, 1e-1),
                                seed=W.SEED_BASE + 4096, mode=1), None, 1
    yield "ragged_sc_momentum", W.custom([9000, 4096, 65, 200000], K=3, period=2, rounds=5,
                                         dist="normal_outliers", scale_range=(1e-3, 1e-1),
                                         seed=W.SEED_BASE + 4097, mode=0), 0.9, 0


def main(out: str) -> int:
    import torch
    from paper_2008_05823_amd import saef
    from paper_2008_05823_amd import workloads as W
    from tests import gpu_harness as H
    print(f"tile-size child: library {saef.LIB_PATH}", flush=True)
    res = {}
    for name, w, mu, mode in cases():
        gs = H.GpuState(w, mu=mu)
        res[f"{name}.n_tiles"] = np.array(gs.layout.info()["n_tiles"])
        for t in range(w.rounds):
            gs.round(t, W.gradients(w, t), mode=mode)
            st = gs.plain(mode=mode)
            for k, v in st.items():
                res[f"{name}.t{t}.{k}"] = np.frombuffer(
                    hashlib.sha256(np.ascontiguousarray(v).tobytes()).digest(), np.uint8)
        for k, v in st.items():
            res[f"{name}.final.{k}"] = v
        assert gs.status() == 0
        print(f"tile-size child: {name} done ({w.rounds} iterations)", flush=True)
    torch.cuda.synchronize()
    np.savez(out, **res)
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1]))
