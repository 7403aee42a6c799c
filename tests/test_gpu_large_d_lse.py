"""GPU parity of the log-sum-exp reductions for 16 < D <= 256 (matrix cores).

a_i = log sum_j exp(g_j - |x_i - y_j|^2 / eps) (the Sinkhorn form), the
Gaussian's log-domain sum log sum_j k_ij exp(g_j) (the same with eps =
2 sigma^2) and the Laplacian's (s = g_j - |x_i - y_j| / sigma, the square root
of the expanded distance), on the fp32 matrix-core kernel: each lane keeps a running
reference and its sums in log2 units, the four lane groups and the column
blocks are merged as (m, s) pairs.  Compared with the fp64 oracle at the
log-sum-exp bar (1e-4 in the log domain beyond the fp32 rounding of a value
of the row maximum's size), with column splits, ragged sizes, spread-out g,
small eps (terms spanning hundreds of binary orders), empty reductions and
block-sparse patterns.
"""
import numpy as np
import pytest

import oracle
from helpers import LSE_TOL, dev, host, lse_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def _data(seed, M, N, D, gspread=1.0, offset=0.0):
    rng = np.random.default_rng(seed)
    x = (offset + rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (offset + rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    g = (gspread * rng.standard_normal((N, 1))).astype(np.float32)
    return x, y, g


CASES = [
    # M, N, D, eps, g spread, offset, col_blocks
    (1, 1, 17, 1.0, 1.0, 0.0, 0),
    (300, 901, 17, 0.5, 1.0, 0.0, 0),
    (513, 1000, 64, 0.05, 2.0, 1.0, 0),     # small eps: terms over hundreds of binary orders
    (257, 777, 100, 1.0, 5.0, 0.0, 3),
    (400, 1200, 128, 0.2, 1.0, 3.0, 1),
    (129, 600, 200, 2.0, 0.5, 0.0, 7),
    # the fp32 expanded form carries an error of about 2^-24 (|x - m|^2 + |y - m|^2) / eps
    # per term in s (m the centre): at D = 256 and eps = 0.01, against squared distances
    # of about 2, that alone is 2e-4 in the log domain, above the bar
    (200, 500, 256, 0.05, 1.0, 0.0, 0),
]


@pytest.mark.parametrize("M,N,D,eps,gs,offset,C", CASES)
def test_sinkhorn_lse_large_d(ctx, M, N, D, eps, gs, offset, C):
    x, y, g = _data(M + N + D, M, N, D, gs, offset)
    out = host(ctx.run("sinkhorn", "lse", dev(x), dev(y), dev(g), eps=eps, col_blocks=C))
    ref, m = oracle.sinkhorn_lse(x, y, g, eps)
    assert out.shape == (M, 1)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


@pytest.mark.parametrize("D,sigma,C", [(20, 0.5, 0), (96, 0.3, 4), (256, 1.0, 0)])
def test_gauss_lse_large_d(ctx, D, sigma, C):
    M, N = 350, 1100
    x, y, g = _data(D, M, N, D)
    out = host(ctx.run("gauss", "lse", dev(x), dev(y), dev(g), sigma=sigma, col_blocks=C))
    ref, m = oracle.kernel_lse("gauss", x, y, g, sigma)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


@pytest.mark.parametrize("D,sigma,C", [(17, 0.5, 0), (64, 0.2, 3), (200, 1.0, 0)])
def test_laplace_lse_large_d(ctx, D, sigma, C):
    # s = g - |x - y| / sigma: g' per column in its own array, sqrt of the expanded d
    M, N = 300, 1000
    x, y, g = _data(D + 5, M, N, D, offset=1.0)
    out = host(ctx.run("laplace", "lse", dev(x), dev(y), dev(g), sigma=sigma, col_blocks=C))
    ref, m = oracle.kernel_lse("laplace", x, y, g, sigma)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def test_lse_large_d_empty_and_ranges(ctx):
    import torch
    from test_gpu_ranges import random_pattern
    x, y, g = _data(5, 700, 900, 40)
    # N = 0: every row is the empty log-sum-exp
    out = host(ctx.run("sinkhorn", "lse", dev(x), torch.zeros((0, 40), device="cuda"),
                       torch.zeros((0, 1), device="cuda"), eps=1.0))
    assert np.isneginf(out).all()
    rng = np.random.default_rng(6)
    rows, ptr, cr = random_pattern(rng, 700, 900, 9, 8)
    for C in (0, 1, 5):
        out = host(ctx.run_ranges("sinkhorn", "lse", dev(x), dev(y), dev(g), dev(rows), dev(ptr),
                                  dev(cr), eps=0.3, col_blocks=C))[:, 0]
        ref, m = oracle.ranges_reduce("lse", x, y, g, rows, ptr, cr, eps=0.3)
        empty = np.isneginf(ref)
        assert np.isneginf(out[empty]).all()
        assert lse_err(out[~empty], ref[~empty], m[~empty]) <= LSE_TOL, C
        out = host(ctx.run_ranges("laplace", "lse", dev(x), dev(y), dev(g), dev(rows), dev(ptr),
                                  dev(cr), sigma=0.4, col_blocks=C))[:, 0]
        ref, m = oracle.ranges_reduce("lse", x, y, g, rows, ptr, cr, formula="laplace", sigma=0.4)
        assert np.isneginf(out[empty]).all()
        assert lse_err(out[~empty], ref[~empty], m[~empty]) <= LSE_TOL, C
