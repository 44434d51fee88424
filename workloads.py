"""Seeded synthetic inputs for the exact-budget LapSum soft top-k.

This module only draws random numbers. It holds none of the method's
arithmetic, so both the float64 oracle and the HIP library can consume its
arrays without sharing any code.

All draws use NumPy's PCG64 (`numpy.random.default_rng`) in float64 and are
cast once to float32. The five workloads mirror the shapes, sizes and value
distributions of the paper's operator benchmarks (synthetic scores, §5 and
Table ks-main) and of its two applications' selection problems (a dense MoE
style batch of routing rows, a megapixel sparse-budget mask):

==========  ============================================================
name        content
==========  ============================================================
single4k    n=4096, r ~ N(0,1), k=16, alpha=-0.5
batch256    256 rows x n=32768, r ~ N(0,1) with 1% exact duplicates per
            row, k=256, alpha=-0.1
n1e6        n=1e6, r ~ N(0,1), k=1000, alpha=-0.05  (full-sort path)
n1e7        n=1e7, r = |x|, x ~ Laplace(0,1), k=2000, alpha=-0.01
            (full-sort and bracketed paths), sample K = ceil(n^(2/3))
n1e8        n=1e8, r = s + e, s ~ N(0,1), e ~ Laplace(0,0.05), k=20000,
            alpha=-0.01 (bracketed path), sample K = 1e5
==========  ============================================================

The bracketed path consumes a table of K Laplace(0, |alpha|) draws (the
"cached kernel noise" of the systematic sampler); it is generated here and
passed to both sides as an input.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = ["Workload", "WORKLOADS", "get", "scores", "upstream_grad",
           "bracket_noise", "default_sample_size", "laplace_noise", "sample_indices"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n: int
    k: float
    alpha: float
    z: float = 5.16
    sample_size: int | None = None   # K for the bracketed path, None = not bracketed
    paths: tuple = ("full",)

    @property
    def t(self) -> float:
        return -self.alpha


def default_sample_size(n: int) -> int:
    """K = ceil(n^(2/3)), computed with integer arithmetic so it is exact."""
    k = int(round(n ** (2.0 / 3.0)))
    while k ** 3 < n ** 2:
        k += 1
    while k > 1 and (k - 1) ** 3 >= n ** 2:
        k -= 1
    return k


WORKLOADS = {
    "single4k": Workload("single4k", 1, 4096, 16.0, -0.5),
    "batch256": Workload("batch256", 256, 32768, 256.0, -0.1),
    "n1e6": Workload("n1e6", 1, 10**6, 1000.0, -0.05),
    "n1e7": Workload("n1e7", 1, 10**7, 2000.0, -0.01,
                     sample_size=default_sample_size(10**7),
                     paths=("full", "bracketed")),
    "n1e8": Workload("n1e8", 1, 10**8, 20000.0, -0.01, sample_size=10**5,
                     paths=("bracketed",)),
}

_SEED = {"single4k": 0, "batch256": 1, "n1e6": 2, "n1e7": 3, "n1e8": 4}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def _rng(name: str, stream: int) -> np.random.Generator:
    s = _SEED[name]
    if name == "single4k" and stream == 0:
        return np.random.default_rng(0)
    return np.random.default_rng([s, stream])


def scores(name: str) -> np.ndarray:
    """float32 scores of shape [batch, n] (C-contiguous)."""
    w = WORKLOADS[name]
    rg = _rng(name, 0)
    if name == "single4k":
        r = rg.standard_normal(w.n).astype(np.float32)
    elif name == "batch256":
        r = rg.standard_normal((w.batch, w.n)).astype(np.float32)
        nd = int(round(0.01 * w.n))
        for row in range(w.batch):
            pos = rg.choice(w.n, 2 * nd, replace=False)
            r[row, pos[:nd]] = r[row, pos[nd:]]
    elif name == "n1e6":
        r = rg.standard_normal(w.n).astype(np.float32)
    elif name == "n1e7":
        r = np.abs(rg.laplace(0.0, 1.0, w.n)).astype(np.float32)
    elif name == "n1e8":
        r = np.empty(w.n, dtype=np.float32)
        # draw in two full-length streams (normal, then Laplace) chunk by
        # chunk to bound host memory; the chunking does not change the draws
        # because each stream gets its own generator state.
        rn = np.random.default_rng([4, 0, 0])
        rl = np.random.default_rng([4, 0, 1])
        step = 1 << 24
        for a in range(0, w.n, step):
            b = min(w.n, a + step)
            r[a:b] = (rn.standard_normal(b - a) + rl.laplace(0.0, 0.05, b - a)).astype(np.float32)
    else:
        raise KeyError(name)
    return np.ascontiguousarray(r.reshape(w.batch, w.n))


def upstream_grad(name: str) -> np.ndarray:
    """float32 upstream gradient dL/dp ~ N(0,1), same shape as the scores."""
    w = WORKLOADS[name]
    if name == "single4k":
        rg = np.random.default_rng([0, 1])
    else:
        rg = _rng(name, 1)
    if w.n * w.batch > (1 << 26):
        out = np.empty(w.batch * w.n, dtype=np.float32)
        step = 1 << 24
        for a in range(0, out.size, step):
            b = min(out.size, a + step)
            out[a:b] = rg.standard_normal(b - a).astype(np.float32)
        return out.reshape(w.batch, w.n)
    return rg.standard_normal((w.batch, w.n)).astype(np.float32)


def laplace_noise(seed, count: int, scale: float) -> np.ndarray:
    """`count` float32 draws of Laplace(0, scale) from default_rng(seed)."""
    return np.random.default_rng(seed).laplace(0.0, scale, count).astype(np.float32)


def sample_indices(seed, n: int, K: int) -> np.ndarray:
    """K indices drawn uniformly from [0, n) with replacement (int32), the
    draws of an i.i.d. bracket sample."""
    return np.random.default_rng(seed).integers(0, n, K).astype(np.int32)


def bracket_noise(name: str) -> np.ndarray:
    """The kernel-noise table eps[K] ~ Laplace(0, |alpha|) for the sampler."""
    w = WORKLOADS[name]
    if w.sample_size is None:
        raise ValueError(f"workload {name} has no bracketed path")
    return laplace_noise([_SEED[name], 2], w.sample_size, w.t)


def random_case(seed: int, n: int, *, dist: str = "normal", ties: float = 0.0,
                batch: int = 1) -> np.ndarray:
    """Small seeded float32 score arrays of various shapes for parity tests.

    dist: normal | laplace_abs | uniform | cauchy | levels16 | lognormal |
          clusters3 | student2 | constant
    ties: fraction of entries overwritten by copies of other entries.
    """
    rg = np.random.default_rng([1000, seed, n, batch])
    shape = (batch, n)
    if dist == "normal":
        x = rg.standard_normal(shape)
    elif dist == "laplace_abs":
        x = np.abs(rg.laplace(0.0, 1.0, shape))
    elif dist == "uniform":
        x = rg.uniform(-1.0, 1.0, shape)
    elif dist == "cauchy":
        x = rg.standard_cauchy(shape)
    elif dist == "levels16":
        x = rg.integers(0, 16, shape).astype(np.float64) / 4.0
    elif dist == "lognormal":
        x = rg.lognormal(0.0, 1.0, shape)
    elif dist == "clusters3":
        c = rg.integers(0, 3, shape)
        x = np.array([-4.0, 0.0, 5.0])[c] + 0.3 * rg.standard_normal(shape)
    elif dist == "student2":
        x = rg.standard_t(2, shape)
    elif dist == "constant":
        x = np.full(shape, 0.75)
    else:
        raise ValueError(dist)
    x = x.astype(np.float32)
    if ties > 0.0 and n > 1:
        nd = int(round(ties * n))
        for row in range(batch):
            if nd == 0:
                break
            nd2 = min(nd, n // 2)
            pos = rg.choice(n, 2 * nd2, replace=False)
            x[row, pos[:nd2]] = x[row, pos[nd2:]]
    return np.ascontiguousarray(x)
