"""GPU parity of the fused Gaussian value + x-gradient for 16 < D <= 256.

The library evaluates it as one Gaussian sum with D + 1 signal columns
[b, b (y - m)] on the matrix cores (64 columns per launch; m a centre of y)
and finishes g_i = (A1_i - (x_i - m) A0_i) / sigma^2.  Compared with the fp64
oracle's gauss_gradx (the definition, any D), normalised per component by the
sum of absolute summands as for the small-D gradient, on both matrix-core
kernels (fp32 products, and the three-way bf16 split), with column splits,
data far from the origin (where the centring matters), one and several
signal chunks, block-sparse patterns, and the Gaussian backward at these D
with scalar cotangents (the fused value + gradient) and with E signal columns
(one Gaussian sum with E (D + 1) columns contracted with the cotangent).
"""
import numpy as np
import pytest

import oracle
from helpers import SUM_TOL, dev, host, norm_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def _data(seed, M, N, D, offset=0.0, E=1):
    # coordinates ~ offset + N(0, 1/D): squared distances of order 2, sigma 1
    rng = np.random.default_rng(seed)
    x = (offset + rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (offset + rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    return x, y, b


CASES = [
    # M, N, D, sigma, offset, col_blocks
    (1, 1, 17, 1.0, 0.0, 0),
    (300, 900, 17, 0.8, 0.0, 0),
    (513, 1000, 64, 1.0, 3.0, 0),        # one chunk of 64 signal columns (D + 1 = 65: two)
    (257, 777, 63, 1.0, 0.0, 3),         # D + 1 = 64: exactly one chunk
    (400, 1200, 128, 1.2, 5.0, 1),
    (129, 600, 200, 1.0, 0.0, 5),
    (200, 500, 256, 1.0, 2.0, 0),        # five chunks, the last of one column
]


@pytest.mark.parametrize("path", ["fp32", "split"])
@pytest.mark.parametrize("M,N,D,sigma,offset,C", CASES)
def test_gradx_large_d_parity(ctx, M, N, D, sigma, offset, C, path):
    from paper_2004_11127_amd import kred
    x, y, b = _data(M + N + D, M, N, D, offset)
    flags = kred.FLAG_DIRECT if path == "fp32" else kred.FLAG_FAST
    out = host(ctx.run("gauss_gradx", "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C,
                       flags=flags))
    ref, norm = oracle.gauss_gradx(x, y, b, sigma)
    assert out.shape == (M, 1 + D)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_gradx_large_d_ranges(ctx):
    from test_gpu_ranges import random_pattern
    rng = np.random.default_rng(4)
    M, N, D = 1200, 1500, 48
    x, y, b = _data(7, M, N, D, offset=1.0)
    rows, ptr, cr = random_pattern(rng, M, N, 12, 9)
    cr = np.concatenate([cr, [[N - 7, N + 30]]]).astype(np.int32)
    ptr = np.concatenate([ptr, [len(cr)]]).astype(np.int32)
    rows = np.concatenate([rows, [[M - 2, M + 9]]]).astype(np.int32)
    for C in (0, 1, 4):
        out = host(ctx.run_ranges("gauss_gradx", "sum", dev(x), dev(y), dev(b), dev(rows), dev(ptr),
                                  dev(cr), sigma=1.0, col_blocks=C))
        ref, norm = oracle.ranges_reduce("gradx", x, y, b, rows, ptr, cr, sigma=1.0)
        assert norm_err(out, ref, norm) <= SUM_TOL, C
        assert (out[norm.sum(1) == 0] == 0).all()


@pytest.mark.parametrize("D,E", [(24, 1), (96, 1), (130, 1)])
def test_backward_large_d_scalar_cotangent(ctx, D, E):
    M, N = 600, 800
    x, y, b = _data(D, M, N, D, offset=0.5, E=E)
    e = np.random.default_rng(D + 1).standard_normal((M, E)).astype(np.float32)
    gx, gy, gb = ctx.gauss_backward(dev(x), dev(y), dev(b), dev(e), sigma=1.0)
    ref, norm = oracle.gauss_vjp(x, y, b, e, 1.0)
    assert norm_err(host(gx), ref, norm) <= SUM_TOL
    ref, norm = oracle.gauss_vjp(y, x, e, b, 1.0)
    assert norm_err(host(gy), ref, norm) <= SUM_TOL
    ref, norm = oracle.kernel_sum("gauss", y, x, e, sigma=1.0)
    assert norm_err(host(gb), ref, norm) <= SUM_TOL


@pytest.mark.parametrize("M,N,D,E,offset", [(500, 700, 64, 6, 0.0), (300, 450, 17, 2, 2.0),
                                             (200, 333, 130, 3, 0.5), (150, 260, 40, 64, 0.0)])
def test_backward_large_d_signal_gradient(ctx, M, N, D, E, offset):
    # E > 1 at large D: gx and gy from the Gaussian sum with the E (D + 1)
    # columns [b_e, b_e (y - m)] contracted with e, gb a Gaussian sum
    x, y, b = _data(3 + E, M, N, D, offset=offset, E=E)
    e = np.random.default_rng(2).standard_normal((M, E)).astype(np.float32)
    gx, gy, gb = ctx.gauss_backward(dev(x), dev(y), dev(b), dev(e), sigma=1.0)
    ref, norm = oracle.gauss_vjp(x, y, b, e, 1.0)
    assert norm_err(host(gx), ref, norm) <= SUM_TOL
    ref, norm = oracle.gauss_vjp(y, x, e, b, 1.0)
    assert norm_err(host(gy), ref, norm) <= SUM_TOL
    ref, norm = oracle.kernel_sum("gauss", y, x, e, sigma=1.0)
    assert norm_err(host(gb), ref, norm) <= SUM_TOL


@pytest.mark.parametrize("E", [1, 3])
def test_backward_ranges_large_d(ctx, E):
    from paper_2004_11127_amd import clusters
    from test_gpu_ranges import random_pattern
    rng = np.random.default_rng(11)
    M, N, D = 900, 1100, 40
    x, y, b = _data(12, M, N, D, offset=0.3, E=E)
    e = rng.standard_normal((M, E)).astype(np.float32)
    pat = random_pattern(rng, M, N, 8, 10)
    tr = clusters.transpose_pattern(*pat, M, N)
    gx, gy, gb = ctx.gauss_backward_ranges(dev(x), dev(y), dev(b), dev(e),
                                           tuple(dev(np.asarray(a, np.int32)) for a in pat),
                                           tuple(dev(a) for a in tr), sigma=1.0)
    rx, nx, ry, ny, rb, nb = oracle.ranges_backward(x, y, b, e, 1.0, *pat)
    assert norm_err(host(gx), rx, nx) <= SUM_TOL
    assert norm_err(host(gy), ry, ny) <= SUM_TOL
    assert norm_err(host(gb), rb, nb) <= SUM_TOL


# With 64 q + 1 signal columns on the 32x32-tile split kernel (D + 1 = 65 or
# 129), the last column is summed on the vector ALU by the first launch; its
# own call then only lets the fp64 contraction run when the guard picks it
@pytest.mark.parametrize("C", [1, 2, 8])
@pytest.mark.parametrize("M,N,D", [(700, 1500, 64), (520, 1100, 128), (300, 65, 64), (1, 1, 64),
                                   (37, 31, 128)])
def test_gradx_last_column_with_the_first_launch(ctx, M, N, D, C):
    from paper_2004_11127_amd import kred
    x, y, b = _data(D + C + N, M, N, D, offset=1.5)
    for _ in range(2):   # the second call finds the first one's partials
        ctx.profile_collect()
        out = host(ctx.run("gauss_gradx", "sum", dev(x), dev(y), dev(b), sigma=1.0, col_blocks=C,
                           flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
        assert ctx.profile_collect()[2] == "mfma_split_kernel"
        ref, norm = oracle.gauss_gradx(x, y, b, 1.0)
        assert norm_err(out, ref, norm) <= SUM_TOL
        # the last coordinate's gradient comes from the extra column alone
        assert norm_err(out[:, -1:], ref[:, -1:], norm[:, -1:]) <= SUM_TOL


def test_vjp_last_column_with_the_first_launch(ctx):
    # E (D + 1) = 3 x 43 = 129 signal columns: the vector-Jacobian product
    from paper_2004_11127_amd import kred
    M, N, D, E = 400, 900, 42, 3
    x, y, b = _data(5, M, N, D, offset=0.5, E=E)
    e = np.random.default_rng(6).standard_normal((M, E)).astype(np.float32)
    gx, gy, gb = ctx.gauss_backward(dev(x), dev(y), dev(b), dev(e), sigma=1.0, flags=kred.FLAG_FAST)
    ref, norm = oracle.gauss_vjp(x, y, b, e, 1.0)
    assert norm_err(host(gx), ref, norm) <= SUM_TOL
    ref, norm = oracle.gauss_vjp(y, x, e, b, 1.0)
    assert norm_err(host(gy), ref, norm) <= SUM_TOL


def test_gradx_last_column_ranges(ctx):
    # block-sparse, D = 64: segments restart the extra column's buffers too;
    # rows in no cluster stay zero
    from paper_2004_11127_amd import kred
    from test_gpu_ranges import random_pattern
    rng = np.random.default_rng(9)
    M, N, D = 900, 1400, 64
    x, y, b = _data(8, M, N, D, offset=1.0)
    rows, ptr, cr = random_pattern(rng, M, N, 10, 8)
    for C in (1, 3):
        out = host(ctx.run_ranges("gauss_gradx", "sum", dev(x), dev(y), dev(b), dev(rows), dev(ptr),
                                  dev(cr), sigma=1.0, col_blocks=C, flags=kred.FLAG_FAST))
        ref, norm = oracle.ranges_reduce("gradx", x, y, b, rows, ptr, cr, sigma=1.0)
        assert norm_err(out, ref, norm) <= SUM_TOL, C
        assert (out[norm.sum(1) == 0] == 0).all()


@pytest.mark.parametrize("C", [1, 4])
def test_gradx_last_column_beyond_the_guard(ctx, C):
    # data past the split kernel's limit: the fp64 contraction takes every
    # launch, the last column's own call included
    from paper_2004_11127_amd import kred
    from test_gpu_large_d_guard import LOG2E, guard_L, limit, two_clusters
    rng = np.random.default_rng(31)
    M, N, D = 300, 800, 64
    x, y = two_clusters(rng, M, N, D, std=0.3 / np.sqrt(D))
    b = rng.standard_normal((N, 1)).astype(np.float32)
    c = 1.05 * limit(D, True) / guard_L(x, y, 1.0)
    sigma = float(np.sqrt(LOG2E / (2 * c)))
    ctx.profile_collect()
    out = host(ctx.run("gauss_gradx", "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == "mfma_f64_kernel"
    ref, norm = oracle.gauss_gradx(x, y, b, sigma)
    assert norm_err(out, ref, norm) <= SUM_TOL
