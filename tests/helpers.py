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
