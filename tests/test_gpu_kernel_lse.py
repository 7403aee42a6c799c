"""GPU parity of the log-domain kernel sums (GAUSS / LAPLACE with the LSE reduction).

a_i = log sum_j k_ij exp(g_j) against the fp64 oracle, |gpu - oracle| <= 1e-4
in the log domain plus fp32 rounding of the row maximum.  The Gaussian runs on
the Sinkhorn-form kernels with eps = 2 sigma^2 (matrix-core exponent when D <=
3 and FLAG_FAST, direct form otherwise); the Laplacian on the direct form.
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


CASES = [
    # formula, M, N, D, sigma, C, path
    ("gauss", 1, 1, 3, 0.3, 0, "fast"),
    ("gauss", 1000, 4099, 3, 0.05, 0, "fast"),
    ("gauss", 700, 2001, 2, 0.02, 3, "fast"),
    ("gauss", 1000, 4099, 3, 0.05, 0, "direct"),
    ("gauss", 300, 1500, 8, 0.3, 5, "direct"),
    ("laplace", 1, 1, 3, 0.3, 0, "direct"),
    ("laplace", 1000, 4099, 3, 0.05, 0, "direct"),
    ("laplace", 513, 777, 1, 0.02, 2, "direct"),
    ("laplace", 257, 1999, 16, 0.5, 7, "direct"),
]


@pytest.mark.parametrize("formula,M,N,D,sigma,C,path", CASES)
def test_kernel_lse_parity(ctx, formula, M, N, D, sigma, C, path):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + N + D)
    x = rng.uniform(0, 1, (M, D)).astype(np.float32)
    y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    g = (3.0 * rng.standard_normal((N, 1))).astype(np.float32)
    flags = kred.FLAG_FAST if path == "fast" else kred.FLAG_DIRECT
    out = host(ctx.run(formula, "lse", dev(x), dev(y), dev(g), sigma=sigma, col_blocks=C,
                       flags=flags))
    ref, m = oracle.kernel_lse(formula, x, y, g, sigma)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


@pytest.mark.parametrize("formula", ["gauss", "laplace"])
def test_kernel_lse_rising_maximum(ctx, formula):
    # log-weights that rise across the columns: the running reference moves
    # by far more than the rescale threshold inside the column range
    rng = np.random.default_rng(2)
    M, N = 500, 5000
    x = rng.uniform(0, 1, (M, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
    g = np.linspace(0.0, 400.0, N).astype(np.float32).reshape(N, 1)
    for C in (0, 3):
        out = host(ctx.run(formula, "lse", dev(x), dev(y), dev(g), sigma=0.1, col_blocks=C))
        ref, m = oracle.kernel_lse(formula, x, y, g, 0.1)
        assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def test_gauss_lse_equals_sinkhorn_form(ctx):
    # the same numbers through the two public pairs: eps = 2 sigma^2
    rng = np.random.default_rng(3)
    x = dev(rng.uniform(0, 1, (2000, 3)).astype(np.float32))
    y = dev(rng.uniform(0, 1, (3000, 3)).astype(np.float32))
    g = dev(rng.standard_normal((3000, 1)).astype(np.float32))
    a = host(ctx.run("gauss", "lse", x, y, g, sigma=0.1))
    b = host(ctx.run("sinkhorn", "lse", x, y, g, eps=0.02))
    np.testing.assert_allclose(a, b, rtol=0, atol=2e-5)


def test_kernel_lse_empty_columns(ctx):
    import torch
    x = dev(np.zeros((5, 3), np.float32))
    y = torch.zeros((0, 3), device="cuda"); g = torch.zeros((0, 1), device="cuda")
    for formula in ("gauss", "laplace"):
        out = host(ctx.run(formula, "lse", x, y, g, sigma=1.0))
        assert out.shape == (5, 1) and np.isneginf(out).all()
