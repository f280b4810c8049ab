"""Reader for the hand-derived worked examples in tests/golden/*.txt."""
from __future__ import annotations

import os

import numpy as np

GOLDEN_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name: str) -> dict:
    out = {}
    with open(os.path.join(GOLDEN_DIR, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, val = line.split(":", 1)
            out[key.strip()] = val.split()
    return out


def floats(vals) -> np.ndarray:
    return np.array([float(v) for v in vals], dtype=np.float32)


def words(vals) -> np.ndarray:
    return np.array([int(v, 0) for v in vals], dtype=np.uint64)


def names() -> list[str]:
    return sorted(f for f in os.listdir(GOLDEN_DIR) if f.endswith(".txt"))
