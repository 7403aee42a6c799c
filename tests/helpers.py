"""Shared test helpers: device transfer and the parity metrics.

Parity bar: for fp32 sums, max |gpu - oracle| / sum_j |F_ij b_j| <= 1e-4 over
checked rows and components (the oracle returns that normaliser); for the
log-sum-exp, |gpu - oracle| <= 1e-4 in the log domain plus fp32 rounding of
the row maximum; for arg-K-min on integer-valued coordinates, identical
indices.
"""
import numpy as np

SUM_TOL = 1e-4
LSE_TOL = 1e-4
TINY_NORM = 1e-30


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def norm_err(gpu, ref, norm):
    """Largest normalised error and the count of rows whose normaliser underflowed."""
    gpu = np.asarray(gpu, dtype=np.float64)
    denom = np.maximum(norm, TINY_NORM)
    return float(np.max(np.abs(gpu - ref) / denom)) if gpu.size else 0.0


def lse_err(gpu, ref, m):
    """Largest log-domain error beyond the fp32 rounding of a value of size |m|."""
    gpu = np.asarray(gpu, dtype=np.float64).reshape(-1)
    allow = LSE_TOL + 4 * np.finfo(np.float32).eps * np.abs(m)
    return float(np.max(np.abs(gpu - ref) - allow)) + LSE_TOL if gpu.size else 0.0


def true_dists(x, y, rows, idx):
    """fp64 squared distances |x_rows[r] - y[idx[r, k]]|^2."""
    xs = x[rows].astype(np.float64)
    ys = y.astype(np.float64)[idx]
    return ((xs[:, None, :] - ys) ** 2).sum(-1)


# The small-D matrix-core path's guard, restated on the host: the kernels run
# it when c R^2 (the squared half-diagonal of the joint bounding box of x and
# y, in coordinates prescaled by sqrt(c)) is at most these limits.
FAST_LIMIT3 = 2048.0        # D <= 3, sums and log-sum-exps
FAST_LIMIT4 = 128.0         # D = 4, sums and log-sum-exps
FAST_LIMIT_NEAREST = 2048.0  # nearest-neighbour forms, every D <= 4
LOG2E = 1.4426950408889634


def fast_scale(formula, reduction, param):
    """sqrt(c) of the matrix-core exponent: c = log2(e) / (2 sigma^2) for the Gaussian
    forms, log2(e) / eps for the Sinkhorn form, 1 for the nearest distances."""
    if formula == "sqdist":
        return 1.0
    if formula == "sinkhorn":
        return float(np.float32(np.sqrt(LOG2E / param)))
    return float(np.float32(np.sqrt(LOG2E / (2.0 * param * param))))


def fast_L(x, y, scale):
    """c R^2 as the guard computes it (fp32)."""
    lo = np.minimum(x.min(0), y.min(0)).astype(np.float32)
    hi = np.maximum(x.max(0), y.max(0)).astype(np.float32)
    h = (np.float32(0.5) * (hi - lo) * np.float32(scale)).astype(np.float32)
    return float(np.sum(h.astype(np.float64) ** 2))


def fast_limit(D, nearest):
    return FAST_LIMIT_NEAREST if nearest else (FAST_LIMIT3 if D <= 3 else FAST_LIMIT4)


def nearest_rank_bound(L, D, dmin):
    """Largest |d(j returned) - d_min| the nearest-neighbour matrix-core path allows.

    The expanded form ranks with an absolute error below 2^-24 (L / 2 + 3 d +
    sqrt(3 d L)) at D <= 3 (plus 8 L 2^-24 at D = 4, from the two products that
    do not fit); a returned index can be off by twice that, and the final
    direct-form fp32 distance adds 4 fp32 roundings of its own size.
    """
    u = 2.0 ** -24
    rank = u * (0.5 * L + 3 * dmin + np.sqrt(3 * dmin * L)) + (8 * u * L if D == 4 else 0.0)
    return 2 * rank + 8 * u * dmin + 1e-30


def grad_err_sigma(gpu, ref, norm, sigma):
    """Gradient error against the benchmark spec's normaliser: sigma |g - ref| / sum_j |k_ij b_j|.

    The gradient in units of the kernel width (d a_i / d(x_i / sigma)) has the
    units of a_i, so the normaliser of the sums applies to it.  gpu and ref are
    M x (1 + D) fused outputs (column 0 the value); norm is the oracle's, whose
    column 0 is sum_j |k_ij b_j|.
    """
    g = np.asarray(gpu, dtype=np.float64)[:, 1:]
    den = np.maximum(norm[:, :1], TINY_NORM)
    return float(np.max(sigma * np.abs(g - ref[:, 1:]) / den)) if g.size else 0.0
