"""GPU parity of the block-sparse Gaussian backward (kred_gauss_backward_ranges).

The oracle builds all three gradients from the row-cluster pattern alone (each
cluster's block through the dense routines, its y- and b-gradients scattered
back onto its columns); the library takes the row-cluster pattern for gx and
its column-side view, built on the host by clusters.transpose_pattern, for gy
and gb.  Every route (matrix-core exponent with a scalar cotangent, the direct
vector-Jacobian kernel with one or several E-slices), forced column chunks,
patterns with gaps, empty clusters and clamped ranges, a truncation rule on
clustered points, and the empty patterns.  Bar: 1e-4 normalised per component
by the sum of absolute summands, as for the dense backward.
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


def random_pattern(rng, M, N, n_rc, n_cc, p_keep=0.4):
    rc = np.sort(rng.choice(np.arange(1, M), 2 * n_rc - 1, replace=False))
    rc = np.concatenate([[0], rc, [M]])
    rows = np.array([[rc[2 * i], rc[2 * i + 1]] for i in range(n_rc)], dtype=np.int32)
    cc = np.concatenate([[0], np.sort(rng.choice(np.arange(1, N), n_cc - 1, replace=False)), [N]])
    ptr, cr = [0], []
    for i in range(n_rc):
        keep = np.nonzero(rng.uniform(size=n_cc) < p_keep)[0]
        cr.extend([cc[k], cc[k + 1]] for k in keep)
        ptr.append(len(cr))
    return rows, np.array(ptr, dtype=np.int32), np.array(cr, dtype=np.int32).reshape(-1, 2)


def _t(a):
    import torch
    a = np.asarray(a, dtype=np.int32)
    return dev(a) if a.size else torch.zeros(a.shape, dtype=torch.int32, device="cuda")


def run_and_check(ctx, x, y, b, e, sigma, pat, flags, C=0, want=(True, True, True)):
    from paper_2004_11127_amd import clusters
    M, N = len(x), len(y)
    tr = clusters.transpose_pattern(*pat, M, N)
    gx, gy, gb = ctx.gauss_backward_ranges(dev(x), dev(y), dev(b), dev(e),
                                           tuple(_t(a) for a in pat), tuple(_t(a) for a in tr),
                                           sigma=sigma, gx=want[0], gy=want[1], gb=want[2],
                                           col_blocks=C, flags=flags)
    rx, nx, ry, ny, rb, nb = oracle.ranges_backward(x, y, b, e, sigma, *pat)
    for got, ref, nrm, name in ((gx, rx, nx, "gx"), (gy, ry, ny, "gy"), (gb, rb, nb, "gb")):
        if got is None:
            continue
        got = host(got)
        err = norm_err(got, ref, nrm)
        assert err <= SUM_TOL, (name, err)
        # rows / columns outside the pattern hold exactly zero
        assert (got[nrm.sum(1) == 0] == 0).all(), name


CASES = [
    # M, N, D, E, sigma, clusters (rows, cols), col_blocks, path
    (3000, 4000, 3, 1, 0.1, (6, 10), 0, "fast"),
    (2000, 2500, 2, 1, 0.05, (40, 30), 3, "fast"),
    (3000, 4000, 3, 1, 0.1, (6, 10), 0, "direct"),
    (1500, 1200, 3, 3, 0.2, (25, 20), 1, "direct"),
    (800, 2000, 5, 17, 0.3, (8, 12), 0, "direct"),
    (1000, 900, 16, 2, 0.5, (12, 9), 5, "direct"),
]


@pytest.mark.parametrize("M,N,D,E,sigma,cl,C,path", CASES)
def test_backward_ranges_parity(ctx, M, N, D, E, sigma, cl, C, path):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + N + D + E)
    x = rng.uniform(0, 1, (M, D)).astype(np.float32)
    y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    e = rng.standard_normal((M, E)).astype(np.float32)
    rows, ptr, cr = random_pattern(rng, M, N, *cl)
    # ranges reaching outside [0, N) and a row cluster past M are clamped
    cr = np.concatenate([cr, [[N - 5, N + 100]]]).astype(np.int32)
    ptr = np.concatenate([ptr, [len(cr)]]).astype(np.int32)
    rows = np.concatenate([rows, [[M - 3, M + 7]]]).astype(np.int32)
    flags = kred.FLAG_FAST if path == "fast" else kred.FLAG_DIRECT
    run_and_check(ctx, x, y, b, e, sigma, (rows, ptr, cr), flags, C)


@pytest.mark.parametrize("want", [(True, False, False), (False, True, False), (False, False, True)])
def test_backward_ranges_single_outputs(ctx, want):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(5)
    x = rng.uniform(0, 1, (900, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (1300, 3)).astype(np.float32)
    b = rng.standard_normal((1300, 2)).astype(np.float32)
    e = rng.standard_normal((900, 2)).astype(np.float32)
    pat = random_pattern(rng, 900, 1300, 9, 11)
    run_and_check(ctx, x, y, b, e, 0.15, pat, kred.FLAG_DIRECT, want=want)


def test_backward_ranges_truncation_rule(ctx):
    # clustered points, sorted by grid cell, pairs within 4 sigma kept
    from paper_2004_11127_amd import clusters, inputs, kred
    w = inputs.mixture_gauss(M=6000, N=7000, D=3, sigma=0.05, seed=3)
    pat = clusters.truncation_pattern(w.x, w.y, cell=0.1, cutoff=0.2)
    x = np.ascontiguousarray(w.x[pat["order_x"]]); y = np.ascontiguousarray(w.y[pat["order_y"]])
    b = np.ascontiguousarray(w.b[pat["order_y"]])
    e = np.random.default_rng(1).standard_normal((len(x), 1)).astype(np.float32)
    p3 = (pat["row_ranges"], pat["col_ptr"], pat["col_ranges"])
    for flags in (kred.FLAG_FAST, kred.FLAG_DIRECT):
        run_and_check(ctx, x, y, b, e, 0.05, p3, flags)


def test_backward_ranges_empty_patterns(ctx):
    import torch
    rng = np.random.default_rng(6)
    x = rng.uniform(0, 1, (300, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (400, 3)).astype(np.float32)
    b = rng.standard_normal((400, 1)).astype(np.float32)
    e = rng.standard_normal((300, 1)).astype(np.float32)
    z2 = torch.zeros((0, 2), dtype=torch.int32, device="cuda")
    z1 = torch.zeros((1,), dtype=torch.int32, device="cuda")
    gx, gy, gb = ctx.gauss_backward_ranges(dev(x), dev(y), dev(b), dev(e), (z2, z1, z2),
                                           (z2, z1, z2), sigma=0.1)
    for g in (gx, gy, gb):
        assert (host(g) == 0).all()
    # clusters without columns, and column clusters without rows
    pat = (np.array([[0, 100], [150, 300]]), np.array([0, 0, 0]), np.zeros((0, 2)))
    run_and_check(ctx, x, y, b, e, 0.1, pat, 0)


def test_backward_ranges_full_pattern_matches_dense(ctx):
    # one cluster over every pair: the dense backward's results
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(8)
    x = rng.uniform(0, 1, (700, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (900, 3)).astype(np.float32)
    b = rng.standard_normal((900, 4)).astype(np.float32)
    e = rng.standard_normal((700, 4)).astype(np.float32)
    pat = (np.array([[0, 700]]), np.array([0, 1]), np.array([[0, 900]]))
    run_and_check(ctx, x, y, b, e, 0.2, pat, kred.FLAG_DIRECT)
