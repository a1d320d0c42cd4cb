"""Seeded synthetic gradients shaped like the paper's workloads.

This module only draws random numbers and describes workload shapes; it holds
none of the codec's arithmetic, so both the GPU path and the CPU oracle can be
fed the same bytes from it.  The paper's datasets and trained models are not
available; these generators stand in for the gradients of the models in the
paper's Table 1 (ResNet-50, NCF) and for two larger models (VGG-16 and a
350M-parameter transformer split into 24 tensors).

Every gradient is drawn with numpy's PCG64 ``default_rng(seed)`` in fp64,
scaled, and rounded to fp32 (round to nearest even).  Large vectors are drawn
in chunks of ``CHUNK`` elements; within a chunk the draws happen in the order
listed in ``_draw_chunk``.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

CHUNK = 1 << 22


@dataclass(frozen=True)
class Workload:
    name: str
    d: int  # total elements of the flat gradient
    n_tensors: int  # coded independently, split like numpy.array_split
    ratio: tuple | None  # (num, den) top-r ratio, or None: every nonzero is selected
    fpr: float  # Bloom filter target false-positive rate
    degree: int  # polynomial degree per segment
    n_seg: int  # requested segments per tensor
    dist: str  # value distribution, see _draw_chunk
    seed: int

    def offsets(self) -> list:
        """Tensor boundaries: numpy.array_split order, so the first d % T
        tensors hold one element more."""
        base, extra = divmod(self.d, self.n_tensors)
        off = [0]
        for t in range(self.n_tensors):
            off.append(off[-1] + base + (1 if t < extra else 0))
        return off


# The five workloads (sizes from the paper's Table 1 where it gives them).
WORKLOADS = {
    w.name: w
    for w in [
        # 1,048,576 values i.i.d. N(0, 1e-3^2); top 1%; FPR 1e-3; degree 5, 1 segment
        Workload("normal_1m", 1_048_576, 1, (1, 100), 1e-3, 5, 1, "normal_1e-3", 1001),
        # ResNet-50-sized flat gradient (25,557,032 parameters), Laplace(0, 5e-4)
        Workload("resnet50_25m", 25_557_032, 1, (1, 100), 1e-3, 5, 8, "laplace_5e-4", 1002),
        # NCF-sized (31,832,577 parameters), 40% exact zeros, N(0, 1e-2^2) elsewhere
        Workload("ncf_32m", 31_832_577, 1, None, 1e-4, 3, 16, "ncf_sparse", 1003),
        # VGG-16-sized (138,357,544), N(0, 1e-3^2) with 0.5% outliers N(0, 0.1^2); top 0.1%
        Workload("vgg16_138m", 138_357_544, 1, (1, 1000), 1e-3, 5, 16, "normal_outliers", 1004),
        # 350M-parameter transformer, 24 tensors, Student-t(3) * 1e-3; top 1% per tensor
        Workload("transformer_355m_x24", 354_823_168, 24, (1, 100), 1e-3, 5, 8, "student_t3", 1005),
        # the 36,864-element ResNet-20 convolution gradient of the paper's Figure 10
        Workload("resnet20_conv_37k", 36_864, 1, (1, 100), 1e-3, 5, 8, "normal_1e-3", 1006),
    ]
}

# Order used by the tests and the benchmark: the first is the small case.
ORDER = ["normal_1m", "resnet50_25m", "ncf_32m", "vgg16_138m", "transformer_355m_x24"]


def _draw_chunk(rng: np.random.Generator, dist: str, n: int) -> np.ndarray:
    if dist == "normal_1e-3":
        x = rng.standard_normal(n) * 1e-3
    elif dist == "laplace_5e-4":
        x = rng.laplace(0.0, 5e-4, n)
    elif dist == "ncf_sparse":
        z = rng.random(n) < 0.4
        x = rng.normal(0.0, 1e-2, n)
        x[z] = 0.0
    elif dist == "normal_outliers":
        x = rng.normal(0.0, 1e-3, n)
        o = rng.random(n) < 0.005
        x[o] = rng.normal(0.0, 0.1, int(o.sum()))
    elif dist == "student_t3":
        x = rng.standard_t(3, n) * 1e-3
    else:
        raise ValueError(dist)
    return x.astype(np.float32)


def generate(w: Workload, out: np.ndarray | None = None) -> np.ndarray:
    """The workload's gradient as contiguous fp32 (same bytes every call)."""
    rng = np.random.default_rng(w.seed)
    g = out if out is not None else np.empty(w.d, dtype=np.float32)
    for s in range(0, w.d, CHUNK):
        e = min(w.d, s + CHUNK)
        g[s:e] = _draw_chunk(rng, w.dist, e - s)
    return g


def generate_prefix(w: Workload, n: int) -> np.ndarray:
    """The first n elements of ``generate(w)`` without drawing the rest."""
    rng = np.random.default_rng(w.seed)
    g = np.empty(n, dtype=np.float32)
    for s in range(0, n, CHUNK):
        full = min(w.d, s + CHUNK) - s
        x = _draw_chunk(rng, w.dist, full)
        e = min(n, s + CHUNK)
        g[s:e] = x[: e - s]
    return g


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).view(np.uint8)).hexdigest()


# ---------------------------------------------------------------------------
# small adversarial inputs for edge cases
# ---------------------------------------------------------------------------


def tied_values(d: int, seed: int) -> np.ndarray:
    """Values from {-2, -1, -0, +0, 1, 2}: ties everywhere, signed zeros."""
    rng = np.random.default_rng(seed)
    pool = np.array([-2.0, -1.0, -0.0, 0.0, 1.0, 2.0], dtype=np.float32)
    return pool[rng.integers(0, pool.size, d)]


def normal(d: int, seed: int, scale: float = 1e-3) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(d) * scale).astype(np.float32)


def sparse_normal(d: int, seed: int, zero_frac: float, scale: float = 1e-2) -> np.ndarray:
    rng = np.random.default_rng(seed)
    z = rng.random(d) < zero_frac
    x = rng.normal(0.0, scale, d)
    x[z] = 0.0
    return x.astype(np.float32)


def random_indices(d: int, n: int, seed: int) -> np.ndarray:
    """n distinct indices in [0, d), ascending."""
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(d, size=n, replace=False)).astype(np.uint32)
