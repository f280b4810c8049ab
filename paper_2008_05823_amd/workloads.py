"""Seeded synthetic SAEF workloads: tensor lists, initial weights, gradients.

This module holds the input generators shared by the tests, the benchmark and
the oracle checks.  It contains none of the method's arithmetic: it only lays
out parameter tensors and draws random numbers.

The paper trains ResNet-56 on CIFAR-100 and ResNet-50 on ImageNet with K = 4
or 8 workers, learning rate 0.1 and layer-wise compression (Experiments,
"CIFAR Settings", "ImageNet Settings", and the method notation list).  Those
datasets and models are not used here: each workload keeps only what the
compression round sees, namely the list of parameter tensor sizes of the model,
the worker count, the averaging period and a per-tensor gradient distribution.

Layout: tensor l starts at a multiple of 64 elements (so a 64-bit sign word
never straddles two tensors); the gap up to the next multiple of 64 is padding
that no kernel touches.  Worker k's vector is row k of a (K, d_pad) array.

Random streams: numpy's SFC64 generator seeded through a SeedSequence of
(seed, stream kind, round t, worker k).  Gradients of round t for worker k come
from their own stream, so any (t, k) can be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

SEED_BASE = 0x5AEF0000

# stream kinds
_K_GRAD, _K_TENSOR_SCALE, _K_X0 = 1, 2, 3


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    K: int                 # simulated workers
    period: int            # error-averaging period p; 0 means never (p = infinity)
    rounds: int            # SAEF iterations in a full run
    tensors: tuple         # ((name, numel), ...) in parameter order
    dist: str              # gradient distribution, see gradient()
    scale_range: tuple     # (lo, hi) of the per-tensor sigma / b, log-uniform
    seed: int
    lr: float = 0.1        # learning rate eta (base lr of both experiments)
    mode: int = 1          # 1 = double-way compression, 0 = single-way

    @property
    def L(self) -> int:
        return len(self.tensors)

    @property
    def sizes(self) -> np.ndarray:
        return np.array([n for _, n in self.tensors], dtype=np.int64)

    @property
    def d(self) -> int:
        return int(self.sizes.sum())

    def layout(self):
        """(offsets, sizes, d_pad): each tensor starts on a 64-element boundary."""
        sizes = self.sizes
        padded = (sizes + 63) // 64 * 64
        offsets = np.concatenate([[0], np.cumsum(padded)[:-1]]).astype(np.int64)
        return offsets, sizes, int(padded.sum())

    @property
    def d_pad(self) -> int:
        return self.layout()[2]

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# --------------------------------------------------------------------------
# parameter tensor lists (parameter order of the usual PyTorch definitions)

def resnet56_cifar_tensors(num_classes: int = 100, width=(16, 32, 64), blocks: int = 9):
    """CIFAR ResNet-56: 3x3 stem, 3 stages x 9 basic blocks, identity (parameter
    free) shortcuts, BN weight and bias after every conv, linear classifier.
    The classifier of the shape list is 64x10 as in the workload definition."""
    t = [("conv1.weight", 3 * 3 * 3 * width[0]),
         ("bn1.weight", width[0]), ("bn1.bias", width[0])]
    c_in = width[0]
    for s, c in enumerate(width):
        for b in range(blocks):
            p = f"layer{s + 1}.{b}"
            t += [(f"{p}.conv1.weight", 3 * 3 * c_in * c),
                  (f"{p}.bn1.weight", c), (f"{p}.bn1.bias", c),
                  (f"{p}.conv2.weight", 3 * 3 * c * c),
                  (f"{p}.bn2.weight", c), (f"{p}.bn2.bias", c)]
            c_in = c
    t += [("fc.weight", width[-1] * num_classes), ("fc.bias", num_classes)]
    return tuple(t)


def resnet50_tensors(num_classes: int = 1000):
    """ImageNet ResNet-50 (bottleneck v1.5): 7x7 stem, stages of 3/4/6/3
    bottlenecks, projection shortcut in the first block of each stage."""
    t = [("conv1.weight", 64 * 3 * 7 * 7), ("bn1.weight", 64), ("bn1.bias", 64)]
    c_in = 64
    for s, (width, nblocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        c_out = width * 4
        for b in range(nblocks):
            p = f"layer{s + 1}.{b}"
            t += [(f"{p}.conv1.weight", c_in * width),
                  (f"{p}.bn1.weight", width), (f"{p}.bn1.bias", width),
                  (f"{p}.conv2.weight", width * width * 9),
                  (f"{p}.bn2.weight", width), (f"{p}.bn2.bias", width),
                  (f"{p}.conv3.weight", width * c_out),
                  (f"{p}.bn3.weight", c_out), (f"{p}.bn3.bias", c_out)]
            if b == 0:
                t += [(f"{p}.downsample.0.weight", c_in * c_out),
                      (f"{p}.downsample.1.weight", c_out),
                      (f"{p}.downsample.1.bias", c_out)]
            c_in = c_out
    t += [("fc.weight", 2048 * num_classes), ("fc.bias", num_classes)]
    return tuple(t)


def bert_base_tensors(vocab: int = 30522, hidden: int = 768, layers: int = 12,
                      ffn: int = 3072, max_pos: int = 512, types: int = 2):
    """BERT-base encoder with separate Q, K, V projections and the pooler."""
    h = hidden
    t = [("embeddings.word", vocab * h), ("embeddings.position", max_pos * h),
         ("embeddings.token_type", types * h),
         ("embeddings.ln.weight", h), ("embeddings.ln.bias", h)]
    for i in range(layers):
        p = f"layer{i}"
        for proj in ("query", "key", "value"):
            t += [(f"{p}.attn.{proj}.weight", h * h), (f"{p}.attn.{proj}.bias", h)]
        t += [(f"{p}.attn.out.weight", h * h), (f"{p}.attn.out.bias", h),
              (f"{p}.attn.ln.weight", h), (f"{p}.attn.ln.bias", h),
              (f"{p}.ffn.in.weight", h * ffn), (f"{p}.ffn.in.bias", ffn),
              (f"{p}.ffn.out.weight", ffn * h), (f"{p}.ffn.out.bias", h),
              (f"{p}.ffn.ln.weight", h), (f"{p}.ffn.ln.bias", h)]
    t += [("pooler.weight", h * h), ("pooler.bias", h)]
    return tuple(t)


# --------------------------------------------------------------------------
# the five workloads

WORKLOADS = {
    "flat64k": Workload("flat64k", K=4, period=5, rounds=10,
                        tensors=(("flat", 65536),), dist="normal",
                        scale_range=(1.0, 1.0), seed=SEED_BASE + 1),
    "resnet56": Workload("resnet56", K=8, period=10, rounds=20,
                         tensors=resnet56_cifar_tensors(num_classes=10),
                         dist="normal", scale_range=(1e-4, 1e-1), seed=SEED_BASE + 2),
    "resnet50": Workload("resnet50", K=8, period=20, rounds=20,
                         tensors=resnet50_tensors(), dist="laplace_zeros",
                         scale_range=(1e-5, 1e-2), seed=SEED_BASE + 3),
    "bert_base": Workload("bert_base", K=16, period=5, rounds=10,
                          tensors=bert_base_tensors(), dist="normal_outliers",
                          scale_range=(1e-4, 1e-1), seed=SEED_BASE + 4),
    "flat256m": Workload("flat256m", K=8, period=5, rounds=5,
                         tensors=(("flat", 1 << 28),), dist="normal",
                         scale_range=(1.0, 1.0), seed=SEED_BASE + 5),
}

ORDER = ["flat64k", "resnet56", "resnet50", "bert_base", "flat256m"]


def get(name: str) -> Workload:
    return WORKLOADS[name]


def custom(sizes, K: int, period: int = 0, rounds: int = 3, dist: str = "normal",
           seed: int = SEED_BASE + 100, mode: int = 1, lr: float = 0.1,
           scale_range=(1.0, 1.0), name: str = "custom") -> Workload:
    """An ad-hoc tensor list (for adversarial sizes in tests)."""
    tensors = tuple((f"t{i}", int(n)) for i, n in enumerate(sizes))
    return Workload(name, K=K, period=period, rounds=rounds, tensors=tensors, dist=dist,
                    scale_range=scale_range, seed=seed, lr=lr, mode=mode)


# --------------------------------------------------------------------------
# random streams

def _rng(w: Workload, kind: int, t: int = 0, k: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([int(w.seed), kind, int(t), int(k)])
    return np.random.Generator(np.random.SFC64(ss))


def tensor_scales(w: Workload) -> np.ndarray:
    """Per-tensor sigma_l (normal) or b_l (Laplace), log-uniform in scale_range,
    drawn once per workload (fixed across rounds and workers)."""
    lo, hi = w.scale_range
    if lo == hi:
        return np.full(w.L, lo, dtype=np.float64)
    u = _rng(w, _K_TENSOR_SCALE).random(w.L)
    return np.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))


def _per_element(w: Workload, per_tensor: np.ndarray) -> np.ndarray:
    """Broadcast one float32 value per tensor to the padded element vector."""
    off, n, d_pad = w.layout()
    out = np.zeros(d_pad, dtype=np.float32)
    for l in range(w.L):
        out[off[l]:off[l] + n[l]] = per_tensor[l]
    return out


def tensor_mask(w: Workload) -> np.ndarray:
    """True on elements that belong to a tensor, False on padding."""
    off, n, d_pad = w.layout()
    m = np.zeros(d_pad, dtype=bool)
    for l in range(w.L):
        m[off[l]:off[l] + n[l]] = True
    return m


def initial_x(w: Workload) -> np.ndarray:
    """x_0 ~ U(-0.05, 0.05) on tensor elements, 0 on padding."""
    d_pad = w.d_pad
    x = _rng(w, _K_X0).random(d_pad, dtype=np.float32) * np.float32(0.1) - np.float32(0.05)
    x[~tensor_mask(w)] = 0.0
    return x


def gradient(w: Workload, t: int, k: int, scales_elem: np.ndarray | None = None) -> np.ndarray:
    """Synthetic stochastic gradient of worker k at round t (float32, d_pad).

    dist:
      normal           N(0, sigma_l^2)
      laplace_zeros    Laplace(0, b_l) with 5% of elements set to exactly 0
      normal_outliers  N(0, sigma_l^2) with 1% of elements replaced by
                       +-100 sigma_l (random sign)
    Padding elements are 0.
    """
    if scales_elem is None:
        scales_elem = _per_element(w, tensor_scales(w).astype(np.float32))
    d_pad = scales_elem.size
    rng = _rng(w, _K_GRAD, t, k)
    if w.dist == "normal":
        g = rng.standard_normal(d_pad, dtype=np.float32)
        g *= scales_elem
    elif w.dist == "laplace_zeros":
        g = rng.standard_exponential(d_pad, dtype=np.float32)
        neg = rng.integers(0, 2, d_pad, dtype=np.uint8).astype(bool)
        np.negative(g, out=g, where=neg)
        g *= scales_elem
        g[rng.random(d_pad, dtype=np.float32) < np.float32(0.05)] = 0.0
    elif w.dist == "normal_outliers":
        g = rng.standard_normal(d_pad, dtype=np.float32)
        g *= scales_elem
        out = rng.random(d_pad, dtype=np.float32) < np.float32(0.01)
        sgn = np.where(rng.integers(0, 2, d_pad, dtype=np.uint8) == 1,
                       np.float32(100.0), np.float32(-100.0))
        g[out] = (sgn * scales_elem)[out]
    else:
        raise ValueError(f"unknown gradient distribution {w.dist!r}")
    g[scales_elem == 0] = 0.0  # padding
    return g


def gradients(w: Workload, t: int, K: int | None = None, threads: int = 1) -> np.ndarray:
    """All K workers' gradients of round t as a (K, d_pad) float32 array;
    threads > 1 draws the workers' streams in parallel (same values: every
    (t, k) has its own stream)."""
    K = w.K if K is None else K
    se = _per_element(w, tensor_scales(w).astype(np.float32))
    out = np.empty((K, se.size), dtype=np.float32)

    def fill(k):
        out[k] = gradient(w, t, k, se)

    if threads > 1 and K > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(min(threads, K)) as ex:
            list(ex.map(fill, range(K)))
    else:
        for k in range(K):
            fill(k)
    return out


def topk_keep(w: Workload, percent: float) -> np.ndarray:
    """Kept elements per tensor for Top-K sparsification at `percent` (the
    paper's Top-1%, 5%, 10%): k_l = ceil(n_l * percent / 100), at least 1.
    Computed in integers (percent in hundredths) so no rounding can move it."""
    hundredths = int(round(percent * 100))
    n = w.sizes
    k = (n * hundredths + 9999) // 10000
    return np.maximum(k, 1).astype(np.int64)


def topk_algorithmic_bytes_per_param(K: int, density: float, mode: int = 1,
                                     averaging: bool = False) -> dict:
    """Bytes the Top-K iteration itself moves per parameter (density = kept
    fraction).  A message is the selection bit (1/8), the rank word share
    (4 B per 64 elements: 1/16) and the kept values (4 density).

    step ahead: read x and e[k], write xh[k]               4 + 8K
    worker: read g[k], e[k]; write e[k]; write the message  (12 + 3/16 + 4 density) K
    server, double-way: read the K messages, read/write e_srv, write the
      server message, update x at the kept elements       K (3/16 + 4 density) + 8 + 3/16
                                                           + 4 density + 8 density
    server, single-way: read the K messages, read/write x  K (3/16 + 4 density) + 8
    an error-averaging round also writes e[k] once more     + 4K
    """
    msg = 3 / 16 + 4 * density
    step = 4 + 8 * K
    worker = (12 + msg) * K
    server = K * msg + (8 + msg + 8 * density if mode == 1 else 8)
    return {"step": step, "worker": worker, "server": server,
            "round": step + worker + server + (4 * K if averaging else 0)}


def algorithmic_bytes_per_param(K: int, mode: int = 1, averaging: bool = False,
                                momentum: bool = False, step_ahead: bool = True,
                                mismatch: bool = False) -> float:
    """Bytes the method itself moves per parameter per round.

    step ahead: read x and e[k], write xh[k]            4 + 8K
    worker compression: read g[k], e[k]; write e[k] and the sign bits   12K + K/8
    server, double-way: read the K sign streams, read/write e_srv and x, write
      the server sign bits                                    16 + 1/8 + K/8
    server, single-way: read the K sign streams, read/write x    8 + K/8
    an error-averaging round also writes e[k] once more          + 4K
    momentum: the worker step also reads and writes m[k]        + 8K
    local error feedback instead of step ahead: read x, write one copy   8
    mismatch bounds: read e[k] and (double-way) e_srv           4K (+ 4)
    """
    step = (4 + 8 * K) if step_ahead else 8
    comp = (20 if momentum else 12) * K + K / 8
    server = (16 + 1 / 8 + K / 8) if mode == 1 else (8 + K / 8)
    mis = (4 * K + (4 if mode == 1 else 0)) if mismatch else 0
    return step + comp + server + (4 * K if averaging else 0) + mis
