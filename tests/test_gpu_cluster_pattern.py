"""GPU construction of the block-sparse truncation pattern (kred_cluster_pattern).

The device builds the grid labels, the stable sort by label, the cluster
ranges and the truncation (Sec. 3 cluster-wise block-sparsity, Sec. 4 block
truncation) and must return exactly the arrays of the host construction
clusters.truncation_pattern: the permutations, row ranges, column pointers,
merged column ranges and the kept-pair count, bit for bit.  Cases: the
block-sparse bench workload (10^6 points, mixture of 8 Gaussians), random
clouds in D = 1..4 with various cells and cutoffs, a single cell, a zero
cutoff, one point, too small a column capacity (overflow reported, nothing
past it written), and the end-to-end block-sparse sum on the device pattern
against the host pattern's.
"""
import numpy as np
import pytest

from helpers import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def _compare(ctx, x, y, cell, cutoff):
    from paper_2004_11127_amd import clusters
    ref = clusters.truncation_pattern(x, y, cell, cutoff)
    t = ctx.cluster_pattern(dev(x), dev(y), cell, cutoff)
    counts = host(t["counts"])
    nr = int(counts[0])
    assert nr == len(ref["row_ranges"])
    assert int(counts[1]) == len(ref["col_ranges"])
    assert int(counts[2]) == ref["pairs"]
    assert int(counts[3]) == 0
    np.testing.assert_array_equal(host(t["order_x"]), ref["order_x"])
    np.testing.assert_array_equal(host(t["order_y"]), ref["order_y"])
    rr = host(t["row_ranges"])
    np.testing.assert_array_equal(rr[:nr], ref["row_ranges"])
    assert (rr[nr:] == len(x)).all()          # padding: empty clusters
    cp = host(t["col_ptr"])
    np.testing.assert_array_equal(cp[:nr + 1], ref["col_ptr"])
    assert (cp[nr + 1:] == cp[nr]).all()
    np.testing.assert_array_equal(host(t["col_ranges"]), ref["col_ranges"])
    return t, ref


def test_bench_workload_pattern(ctx):
    # the block-sparse bench workload: cells of 2 sigma, truncation at 6 sigma
    from paper_2004_11127_amd import inputs
    w = inputs.mixture_gauss(M=1_000_000, N=1_000_000, D=3, sigma=0.05, seed=0)
    _compare(ctx, w.x, w.y, 2.0 * w.sigma, 6.0 * w.sigma)


@pytest.mark.parametrize("D,M,N,cell,cutoff,seed", [
    (1, 5000, 7000, 0.01, 0.05, 1),
    (2, 3000, 4000, 0.05, 0.2, 2),
    (3, 20000, 15000, 0.1, 0.3, 3),
    (3, 4000, 5000, 0.37, 0.0, 4),      # zero cutoff: only cells within one diagonal
    (4, 6000, 3000, 0.25, 0.6, 5),
    (3, 777, 9999, 0.03, 0.11, 6),      # many clusters, most with one point
])
def test_random_patterns(ctx, D, M, N, cell, cutoff, seed):
    rng = np.random.default_rng(seed)
    x = rng.uniform(-1, 2, (M, D)).astype(np.float32)
    y = (0.5 * rng.standard_normal((N, D)) + 0.3).astype(np.float32)
    _compare(ctx, x, y, cell, cutoff)


def test_degenerate_patterns(ctx):
    rng = np.random.default_rng(9)
    x = rng.uniform(0, 1, (500, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (800, 3)).astype(np.float32)
    _compare(ctx, x, y, 10.0, 1.0)                        # one cell for everything
    _compare(ctx, x[:1], y[:1], 0.1, 0.2)                 # one point each
    _compare(ctx, np.repeat(x[:3], 100, 0), y, 0.05, 0.1)  # many equal points (stable order)


def test_overflow_is_reported(ctx):
    from paper_2004_11127_amd import clusters
    rng = np.random.default_rng(12)
    x = rng.uniform(0, 1, (3000, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (3000, 3)).astype(np.float32)
    ref = clusters.truncation_pattern(x, y, 0.05, 0.1)
    nnz = len(ref["col_ranges"])
    cap = nnz // 2
    t = ctx.cluster_pattern(dev(x), dev(y), 0.05, 0.1, col_cap=cap)
    counts = host(t["counts"])
    assert int(counts[1]) == nnz and int(counts[3]) == 1
    # the ranges below the capacity are the right ones
    np.testing.assert_array_equal(host(t["col_ranges"]), ref["col_ranges"][:cap])


def test_rejects_bad_arguments(ctx):
    import torch
    from paper_2004_11127_amd import kred
    x = dev(np.zeros((10, 3), np.float32))
    with pytest.raises(kred.KredError):
        ctx.cluster_pattern(x, x, 0.0, 1.0)
    with pytest.raises(kred.KredError):
        ctx.cluster_pattern(x, x, 0.1, -1.0)
    with pytest.raises(kred.KredError):
        ctx.cluster_pattern(dev(np.zeros((10, 9), np.float32)), dev(np.zeros((10, 9), np.float32)),
                            0.1, 1.0)


def test_gather_rows_round_trip(ctx):
    import torch
    rng = np.random.default_rng(21)
    a = rng.standard_normal((5000, 3)).astype(np.float32)
    perm = rng.permutation(5000).astype(np.int32)
    g = host(ctx.gather_rows(dev(a), dev(perm)))
    np.testing.assert_array_equal(g, a[perm])
    back = host(ctx.gather_rows(dev(g), dev(perm), inverse=True))
    np.testing.assert_array_equal(back, a)


def test_block_sparse_sum_on_the_device_pattern(ctx):
    # the whole block-sparse pipeline on the device: pattern, gathers, the
    # block-sparse Gaussian sum (nr = M, the padded clusters empty, so the
    # count is never read back), the inverse gather; against the same sum on
    # the host pattern
    import oracle
    from helpers import SUM_TOL, norm_err
    from paper_2004_11127_amd import clusters, kred
    rng = np.random.default_rng(31)
    M, N, sigma = 6000, 8000, 0.05
    centres = rng.uniform(0, 1, (6, 3))
    x = (centres[rng.integers(0, 6, M)] + 0.05 * rng.standard_normal((M, 3))).astype(np.float32)
    y = (centres[rng.integers(0, 6, N)] + 0.05 * rng.standard_normal((N, 3))).astype(np.float32)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    t = ctx.cluster_pattern(dev(x), dev(y), 2 * sigma, 6 * sigma)
    xs = ctx.gather_rows(dev(x), t["order_x"])
    ys = ctx.gather_rows(dev(y), t["order_y"])
    bs = ctx.gather_rows(dev(b), t["order_y"])
    out_s = ctx.run_ranges("gauss", "sum", xs, ys, bs, t["row_ranges"], t["col_ptr"],
                           t["col_ranges"], sigma=sigma)
    out = host(ctx.gather_rows(out_s, t["order_x"], inverse=True))
    ref = clusters.truncation_pattern(x, y, 2 * sigma, 6 * sigma)
    xo, yo, bo = x[ref["order_x"]], y[ref["order_y"]], b[ref["order_y"]]
    want, norm = oracle.ranges_reduce("sum", xo, yo, bo, ref["row_ranges"], ref["col_ptr"],
                                      ref["col_ranges"], formula="gauss", sigma=sigma)
    got_sorted = out[ref["order_x"]]
    assert norm_err(got_sorted, want, norm) <= SUM_TOL
