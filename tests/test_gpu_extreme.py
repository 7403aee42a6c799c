"""GPU parity of the min / max / arg-min / arg-max and K-min reductions against the fp64 oracle.

Exact cases use integer coordinates (and integer b), where every distance and
product is exact in fp32 and ties abound: values and indices (lowest index on
ties) must match the oracle bit for bit, on the direct kernels (D <= 16) and
on the matrix-core arg-K-min lists (D > 16).  On real-valued data the values
must agree to 1e-4 of the row's scale max_j |F_ij| and each returned index
must be a valid arg-extreme: F at that index within the same tolerance of the
extreme value (fp32 and fp64 may order near-ties differently).
"""
import numpy as np
import pytest

import oracle
from helpers import dev, fast_L, host, nearest_rank_bound

pytestmark = pytest.mark.gpu
TOL = 1e-4
TINY = 2.0 ** -120   # fp32 flushes kernel values below this to zero


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def _ints(rng, n, D, lo=-3, hi=4):
    return rng.integers(lo, hi, (n, D)).astype(np.float32)


def _f_at(formula, x, y, b, idx, param):
    """F_ij (fp64) at the given column index per row and component."""
    x64, y64 = x.astype(np.float64), y.astype(np.float64)
    E = idx.shape[1]
    out = np.empty(idx.shape)
    for e in range(E):
        j = idx[:, e]
        d = ((x64 - y64[j]) ** 2).sum(1)
        if formula == "sinkhorn":
            out[:, e] = b[j, 0].astype(np.float64) - d / param
        elif b is None:
            out[:, e] = d
        else:
            k = {"gauss": np.exp(-d / (2 * param ** 2)), "laplace": np.exp(-np.sqrt(d) / param),
                 "sqdist": d}[formula]
            out[:, e] = k * b[j, e].astype(np.float64)
    return out


OPS = {"min": ("min", False), "max": ("max", False), "argmin": ("min", True), "argmax": ("max", True)}

EXACT = [
    # M, N, D, C
    (1, 1, 3, 0), (300, 1000, 1, 0), (700, 2049, 3, 3), (257, 999, 8, 1), (129, 4000, 16, 16),
]


@pytest.mark.parametrize("M,N,D,C", EXACT)
@pytest.mark.parametrize("red", ["min", "max", "argmin", "argmax"])
def test_sqdist_extreme_exact(ctx, M, N, D, C, red):
    rng = np.random.default_rng(M + N + D)
    x, y = _ints(rng, M, D), _ints(rng, N, D)
    out = host(ctx.run("sqdist", red, dev(x), dev(y), None, col_blocks=C))
    op, arg = OPS[red]
    val, idx, _ = oracle.extreme("sqdist", op, x, y)
    if arg:
        np.testing.assert_array_equal(out, idx.astype(np.int32))
    else:
        np.testing.assert_array_equal(out, val.astype(np.float32))


@pytest.mark.parametrize("M,N,D,C", [(300, 2000, 32, 0), (129, 5000, 64, 3), (1000, 1500, 100, 0)])
@pytest.mark.parametrize("red", ["min", "argmin"])
def test_sqdist_min_large_d_exact(ctx, M, N, D, C, red):
    # D > 16: read off the matrix-core arg-K-min lists with K = 1
    rng = np.random.default_rng(D + C)
    x, y = _ints(rng, M, D, -8, 9), _ints(rng, N, D, -8, 9)
    out = host(ctx.run("sqdist", red, dev(x), dev(y), None, col_blocks=C))
    val, idx, _ = oracle.extreme("sqdist", "min", x, y)
    ref = idx.astype(np.int32) if red == "argmin" else val.astype(np.float32)
    np.testing.assert_array_equal(out, ref)


@pytest.mark.parametrize("M,N,D,K,C", [(200, 1000, 3, 1, 0), (300, 2049, 3, 10, 3), (129, 700, 16, 16, 1),
                                       (100, 3000, 8, 64, 0), (257, 4000, 64, 10, 0), (64, 500, 33, 5, 7)])
def test_kmin_exact(ctx, M, N, D, K, C):
    rng = np.random.default_rng(K + D)
    x, y = _ints(rng, M, D, -4, 5), _ints(rng, N, D, -4, 5)
    vals = host(ctx.run("sqdist", "kmin", dev(x), dev(y), None, K=K, col_blocks=C))
    idx = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=K, col_blocks=C))
    ridx, rdist = oracle.argkmin(x, y, K)
    np.testing.assert_array_equal(vals, rdist.astype(np.float32))
    np.testing.assert_array_equal(idx, ridx.astype(np.int32))


@pytest.mark.parametrize("red", ["min", "max", "argmin", "argmax"])
def test_sqdist_with_integer_b_exact(ctx, red):
    rng = np.random.default_rng(3)
    x, y = _ints(rng, 500, 3), _ints(rng, 1500, 3)
    b = rng.integers(-3, 4, (1500, 5)).astype(np.float32)
    out = host(ctx.run("sqdist", red, dev(x), dev(y), dev(b), col_blocks=4))
    op, arg = OPS[red]
    val, idx, _ = oracle.extreme("sqdist", op, x, y, b)
    np.testing.assert_array_equal(out, idx.astype(np.int32) if arg else val.astype(np.float32))


REAL = [
    # formula, M, N, D, E, param, C
    ("gauss", 500, 2000, 3, 1, 0.1, 0),
    ("gauss", 300, 1500, 2, 3, 0.2, 3),
    ("gauss", 129, 999, 8, 16, 0.5, 1),
    ("gauss", 100, 700, 3, 20, 0.1, 0),
    ("laplace", 400, 1200, 5, 4, 0.3, 2),
    ("sqdist", 333, 1234, 12, 2, 1.0, 0),
    ("sinkhorn", 600, 2500, 3, 1, 0.01, 0),
    ("sinkhorn", 257, 1000, 16, 1, 0.5, 5),
    # 16 < D <= 256: the fp32 matrix-core kernel, signal columns in slices of 16
    ("gauss", 300, 1000, 32, 1, 1.5, 0),
    ("gauss", 200, 800, 64, 20, 2.0, 3),
    ("laplace", 257, 900, 100, 3, 2.0, 1),
    ("sqdist", 200, 700, 40, 2, 1.0, 0),
    ("sinkhorn", 300, 1200, 48, 1, 4.0, 0),
    ("sinkhorn", 129, 600, 256, 1, 20.0, 5),
]


@pytest.mark.parametrize("formula,M,N,D,E,param,C", REAL)
@pytest.mark.parametrize("red", ["min", "max", "argmin", "argmax"])
def test_extreme_real_data(ctx, formula, M, N, D, E, param, C, red):
    rng = np.random.default_rng(M * 3 + N + E)
    x = rng.uniform(0, 1, (M, D)).astype(np.float32)
    y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    kw = dict(eps=param) if formula == "sinkhorn" else dict(sigma=param)
    out = host(ctx.run(formula, red, dev(x), dev(y), dev(b), col_blocks=C, **kw))
    op, arg = OPS[red]
    val, idx, scale = oracle.extreme(formula, op, x, y, b, param=param)
    allow = TOL * scale + TINY * np.abs(b).max()
    if arg:
        assert out.dtype == np.int32 and out.min() >= 0 and out.max() < N
        f = _f_at(formula, x, y, b, out.astype(np.int64), param)
        assert (np.abs(f - val) <= allow).all()
        assert (out == idx).mean() > 0.99   # near-ties aside, the same index
    else:
        assert (np.abs(out.astype(np.float64) - val) <= allow).all()


@pytest.mark.parametrize("D,C", [(24, 0), (128, 4)])
@pytest.mark.parametrize("red", ["max", "argmax"])
def test_farthest_point_large_d(ctx, D, C, red):
    # the squared distance's max without b at D > 16 (one signal column of ones)
    rng = np.random.default_rng(D + C)
    x = rng.uniform(0, 1, (300, D)).astype(np.float32)
    y = rng.uniform(0, 1, (1100, D)).astype(np.float32)
    out = host(ctx.run("sqdist", red, dev(x), dev(y), None, col_blocks=C))
    val, idx, scale = oracle.extreme("sqdist", "max", x, y)
    allow = TOL * scale
    if red == "argmax":
        f = _f_at("sqdist", x, y, None, out.astype(np.int64), 1.0)
        assert (np.abs(f - val) <= allow).all()
        assert (out == idx).mean() > 0.99
    else:
        assert (np.abs(out.astype(np.float64) - val) <= allow).all()


def test_extreme_large_d_ranges(ctx):
    from test_gpu_ranges import random_pattern
    rng = np.random.default_rng(31)
    M, N, D = 900, 1300, 48
    x = rng.uniform(0, 1, (M, D)).astype(np.float32)
    y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, 2)).astype(np.float32)
    pat = random_pattern(rng, M, N, 9, 11)
    for red in ("max", "argmin"):
        for C in (0, 1, 4):
            out = host(ctx.run_ranges("gauss", red, dev(x), dev(y), dev(b), dev(pat[0]), dev(pat[1]),
                                      dev(pat[2]), sigma=2.0, col_blocks=C))
            ref, aux = oracle.ranges_reduce(red.replace("arg", ""), x, y, b, *pat, formula="gauss",
                                            param=2.0)
            empty = aux < 0
            if red == "argmin":
                assert (out[empty] == -1).all()
                # a valid arg-min where the reference has one
                assert (out[~empty] == aux[~empty]).mean() > 0.99
            else:
                assert np.isneginf(out[empty]).all()
                assert np.abs(out[~empty] - ref[~empty]).max() <= 1e-4 * np.abs(b).max()


@pytest.mark.parametrize("red,fill", [("min", np.inf), ("max", -np.inf), ("argmin", -1), ("argmax", -1)])
def test_extreme_empty_columns(ctx, red, fill):
    import torch
    x = dev(np.zeros((7, 3), np.float32)); y = torch.zeros((0, 3), device="cuda")
    out = host(ctx.run("sqdist", red, x, y, None))
    assert out.shape == (7, 1) and (out == fill).all()
    b = torch.zeros((0, 2), device="cuda")
    out = host(ctx.run("gauss", red, x, y, b, sigma=1.0))
    assert out.shape == (7, 2) and (out == fill).all()


def test_extreme_deterministic_and_profiled(ctx):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(9)
    x = dev(rng.uniform(0, 1, (3000, 3)).astype(np.float32))
    y = dev(rng.uniform(0, 1, (5000, 3)).astype(np.float32))
    b = dev(rng.standard_normal((5000, 2)).astype(np.float32))
    ctx.profile_collect()
    r1 = host(ctx.run("gauss", "argmax", x, y, b, sigma=0.05, flags=kred.FLAG_PROFILE))
    n, ms, name = ctx.profile_collect()
    assert n == 1 and name == "extreme_kernel"
    r2 = host(ctx.run("gauss", "argmax", x, y, b, sigma=0.05))
    np.testing.assert_array_equal(r1, r2)


FAST_NN = [
    # M, N, D, C
    (1, 1, 3, 0), (700, 2049, 3, 3), (3000, 5000, 2, 0), (1500, 999, 1, 16),
    (700, 2049, 4, 3), (3000, 5000, 4, 0),
]


@pytest.mark.parametrize("M,N,D,C", FAST_NN)
@pytest.mark.parametrize("red", ["min", "argmin", "argkmin1"])
def test_nearest_fast_path_exact(ctx, M, N, D, C, red):
    # D <= 4 with KRED_FLAG_FAST: the distance comes from the matrix cores (exact
    # on integer coordinates); min / arg-min / arg-K-min with K = 1 must match
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + N + D + C)
    x, y = _ints(rng, M, D, -20, 21), _ints(rng, N, D, -20, 21)
    if red == "argkmin1":
        out = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=1, col_blocks=C,
                           flags=kred.FLAG_FAST))
    else:
        out = host(ctx.run("sqdist", red, dev(x), dev(y), None, col_blocks=C, flags=kred.FLAG_FAST))
    val, idx, _ = oracle.extreme("sqdist", "min", x, y)
    if red == "min":
        np.testing.assert_array_equal(out, val.astype(np.float32))
    else:
        np.testing.assert_array_equal(out, idx.astype(np.int32))


def test_nearest_fast_path_real_data(ctx):
    # real-valued mixture data: the distance and a valid nearest index
    from paper_2004_11127_amd import inputs, kred
    w = inputs.mixture_gauss(M=20000, N=30000, D=3, sigma=0.05, seed=3)
    d = host(ctx.run("sqdist", "min", dev(w.x), dev(w.y), None, flags=kred.FLAG_FAST))
    j = host(ctx.run("sqdist", "argmin", dev(w.x), dev(w.y), None, flags=kred.FLAG_FAST))
    val, idx, scale = oracle.extreme("sqdist", "min", w.x, w.y)
    # every row: the returned index's distance, and the returned value, within
    # the expanded form's ranking bound of the true nearest distance (the
    # matrix cores rank; the final candidates' distances are direct-form fp32)
    allow = nearest_rank_bound(fast_L(w.x, w.y, 1.0), 3, val)
    f = _f_at("sqdist", w.x, w.y, None, j.astype(np.int64), 1.0)
    assert (np.abs(f - val) <= allow).all()
    assert (np.abs(d.astype(np.float64) - val) <= allow).all()
    # (an index differs from the oracle's only between points whose distances
    # are within the bound: the check on f above covers it)
    assert ((j == idx) | (np.abs(f - val) <= allow)).all()


def test_nearest_fast_kernel_is_used_and_falls_back(ctx):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(12)
    x = rng.uniform(0, 1, (3000, 3)).astype(np.float32); y = rng.uniform(0, 1, (3000, 3)).astype(np.float32)
    ctx.profile_collect()
    ctx.run("sqdist", "min", dev(x), dev(y), None, flags=kred.FLAG_FAST | kred.FLAG_PROFILE)
    assert ctx.profile_collect()[2] == "fast_kernel"
    # data far outside the accuracy guard (half-diagonal 86): the direct kernel answers
    xs, ys = x * 100.0, y * 100.0
    d = host(ctx.run("sqdist", "min", dev(xs), dev(ys), None, flags=kred.FLAG_FAST))
    val, _, scale = oracle.extreme("sqdist", "min", xs, ys)
    assert (np.abs(d.astype(np.float64) - val) <= TOL * scale).all()


FAST_KNN = [
    # M, N, D, K, C
    (700, 2049, 3, 4, 3), (3000, 5000, 2, 10, 0), (1500, 999, 1, 16, 16), (257, 4000, 3, 7, 0),
    (1000, 1500, 3, 12, 1), (64, 64, 3, 16, 0),
    (700, 2049, 4, 10, 3), (1000, 1500, 4, 16, 0), (500, 800, 4, 4, 1),
]


@pytest.mark.parametrize("M,N,D,K,C", FAST_KNN)
@pytest.mark.parametrize("red", ["argkmin", "kmin"])
def test_knn_fast_path_exact(ctx, M, N, D, K, C, red):
    # D <= 4, 1 < K <= 16 with KRED_FLAG_FAST: distances from the matrix cores (exact on
    # integer coordinates inside the guard), per-lane lists merged by (distance, index)
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + N + D + K + C)
    x, y = _ints(rng, M, D, -20, 21), _ints(rng, N, D, -20, 21)
    y[N // 2:N // 2 + N // 8] = y[:N // 8]   # exact ties between columns
    ctx.profile_collect()
    out = host(ctx.run("sqdist", red, dev(x), dev(y), None, K=K, col_blocks=C,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == "fast_kernel"
    idx, dist = oracle.argkmin(x, y, K)
    if red == "argkmin":
        np.testing.assert_array_equal(out, idx.astype(np.int32))
    else:
        np.testing.assert_array_equal(out, dist.astype(np.float32))


def test_knn_fast_path_real_data(ctx):
    # real-valued mixture data: distances within the tolerance, valid indices
    from paper_2004_11127_amd import inputs, kred
    w = inputs.mixture_gauss(M=20000, N=30000, D=3, sigma=0.05, seed=4)
    K = 10
    idx = host(ctx.run("sqdist", "argkmin", dev(w.x), dev(w.y), None, K=K, flags=kred.FLAG_FAST))
    kd = host(ctx.run("sqdist", "kmin", dev(w.x), dev(w.y), None, K=K, flags=kred.FLAG_FAST))
    rows = np.sort(np.random.default_rng(1).choice(20000, 500, replace=False))
    ridx, rdist = oracle.argkmin(w.x, w.y, K, rows=rows)
    # the matrix cores only rank; the returned distances are direct-form fp32,
    # accurate relative to themselves (not only to the row's largest distance)
    rel = 1e-5 * rdist + 1e-12
    assert (np.abs(kd[rows].astype(np.float64) - rdist) <= rel).all()
    got = ((w.x[rows, None, :].astype(np.float64) - w.y[idx[rows]].astype(np.float64)) ** 2).sum(-1)
    assert (np.abs(got - rdist) <= rel).all()
    # fp32 and fp64 may order near-ties among the K-th neighbours differently
    assert (idx[rows] == ridx).mean() > 0.999


def test_knn_fast_path_falls_back_on_wide_data(ctx):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(6)
    x = _ints(rng, 800, 3, -300, 300); y = _ints(rng, 1200, 3, -300, 300)   # R^2 >> 2048
    out = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=6, flags=kred.FLAG_FAST))
    np.testing.assert_array_equal(out, oracle.argkmin(x, y, 6)[0].astype(np.int32))
