"""Seeded synthetic inputs for the kred workloads.

Random draws only: this module holds none of the reductions' arithmetic.  The
GPU library and the oracle both read what it returns, so both see identical
fp32 arrays.  Every workload draws from ``numpy.random.default_rng(seed)``
(PCG64) in a fixed order and casts to float32 at the end.

The paper's benchmark (Sec. 3, table) is the Gaussian sum of Eq. (1) on
synthetic point clouds with M = N and D = 3 in float32; it states no
distribution, so the workloads below fix one each.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class Workload:
    name: str
    formula: str            # "gauss" | "laplace" | "sqdist" | "gauss_gradx" | "sinkhorn"
    reduction: str          # "sum" | "lse" | "argkmin"
    x: np.ndarray           # (M, D) float32
    y: np.ndarray           # (N, D) float32
    b: np.ndarray | None    # (N, E) float32, or None for arg-K-min
    sigma: float = 1.0
    eps: float = 1.0
    K: int = 0
    meta: dict = field(default_factory=dict)

    @property
    def M(self):
        return self.x.shape[0]

    @property
    def N(self):
        return self.y.shape[0]

    @property
    def D(self):
        return self.x.shape[1]

    @property
    def E(self):
        return 0 if self.b is None else self.b.shape[1]


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def uniform_gauss(M=10_000, N=10_000, D=3, E=1, sigma=0.1, seed=0):
    """x, y ~ U[0,1]^D, b ~ N(0,1)^E; Gaussian sum (10k x 10k, D=3, sigma=0.1 by default)."""
    rng = np.random.default_rng(seed)
    x = rng.uniform(0.0, 1.0, (M, D))
    y = rng.uniform(0.0, 1.0, (N, D))
    b = rng.standard_normal((N, E))
    return Workload("gauss_sum_uniform", "gauss", "sum", _f32(x), _f32(y), _f32(b), sigma=sigma,
                    meta=dict(dist="uniform[0,1]^D", seed=seed))


def mixture_points(rng, n_points, centres, std):
    labels = rng.integers(0, centres.shape[0], n_points)
    return centres[labels] + std * rng.standard_normal((n_points, centres.shape[1]))


def mixture_gauss(M=1_000_000, N=1_000_000, D=3, sigma=0.05, n_centres=8, std=0.05, seed=0,
                  formula="gauss_gradx"):
    """x, y from one mixture of n_centres isotropic Gaussians (std 0.05, centres U[0,1]^D),
    drawn independently; b ~ N(0,1).  Default: the 1e6 x 1e6 Gaussian sum with x-gradient."""
    rng = np.random.default_rng(seed)
    centres = rng.uniform(0.0, 1.0, (n_centres, D))
    x = mixture_points(rng, M, centres, std)
    y = mixture_points(rng, N, centres, std)
    b = rng.standard_normal((N, 1))
    return Workload("%s_mixture" % formula, formula, "sum", _f32(x), _f32(y), _f32(b),
                    sigma=sigma, meta=dict(dist="mixture of %d Gaussians, std %g" % (n_centres, std),
                                           seed=seed))


def sinkhorn_lse(M=1_000_000, N=1_000_000, D=3, eps=0.01, shift=0.3, seed=0):
    """x ~ U[0,1]^D, y ~ U[0,1]^D + shift e_0, g ~ N(0,1); log-sum-exp with eps."""
    rng = np.random.default_rng(seed)
    x = rng.uniform(0.0, 1.0, (M, D))
    y = rng.uniform(0.0, 1.0, (N, D))
    y[:, 0] += shift
    g = rng.standard_normal((N, 1))
    return Workload("sinkhorn_lse", "sinkhorn", "lse", _f32(x), _f32(y), _f32(g), eps=eps,
                    meta=dict(dist="uniform, y shifted by %g in dim 0" % shift, seed=seed))


def highdim_gauss(M=200_000, N=200_000, D=128, E=16, sigma=1.0, seed=0):
    """x, y ~ N(0, I/D), b ~ N(0,1)^E; high-dimensional Gaussian sum with a vector signal."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, D)) / np.sqrt(D)
    y = rng.standard_normal((N, D)) / np.sqrt(D)
    b = rng.standard_normal((N, E))
    return Workload("gauss_sum_highdim", "gauss", "sum", _f32(x), _f32(y), _f32(b), sigma=sigma,
                    meta=dict(dist="N(0, I/%d)" % D, seed=seed))


def integer_knn(M=100_000, N=1_000_000, D=64, K=10, n_centres=32, std=3.0, lo=-8, hi=8, seed=0):
    """Integer-valued points: n_centres integer centres in [lo,hi]^D, points = centre +
    std N(0,1), rounded and clipped to [lo,hi], stored as float32; arg-K-min with K."""
    rng = np.random.default_rng(seed)
    centres = rng.integers(lo, hi + 1, (n_centres, D)).astype(np.float64)
    x = np.clip(np.rint(mixture_points(rng, M, centres, std)), lo, hi)
    y = np.clip(np.rint(mixture_points(rng, N, centres, std)), lo, hi)
    return Workload("sqdist_argkmin_integer", "sqdist", "argkmin", _f32(x), _f32(y), None, K=K,
                    meta=dict(dist="integer mixture of %d Gaussians, std %g, clip [%d,%d]"
                              % (n_centres, std, lo, hi), seed=seed))


def sample_rows(M, S=1024, seed=12345):
    """S distinct row indices in [0, M), sorted (all rows when M <= S)."""
    if M <= S:
        return np.arange(M, dtype=np.int64)
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(M, S, replace=False)).astype(np.int64)


# The five workloads (sizes as used by the parity tests and the benchmark).
def workload(name, **kw):
    table = {
        "c1": lambda: uniform_gauss(**kw),
        "c2": lambda: mixture_gauss(**kw),
        "c3": lambda: sinkhorn_lse(**kw),
        "c4": lambda: highdim_gauss(**kw),
        "c5": lambda: integer_knn(**kw),
    }
    return table[name]()
