"""GPU parity of block-sparse (cluster-wise) reductions, kred_run_ranges, against the oracle.

Row cluster I reduces over its own list of column ranges only; rows in no
cluster, and clusters without columns, hold the empty reduction.  Patterns are
random (gaps between row clusters, clusters with no column ranges, clusters
spanning several workgroups, hundreds of clusters for the device-side block
map) plus ranges that need clamping to [0, M) x [0, N).  Same bars as the
dense tests: normalised 1e-4 for sums, 1e-4 in the log domain for
log-sum-exp, bit-exact values and indices on integer data for the
arg-K-min / K-min / min / max families.
"""
import numpy as np
import pytest

import oracle
from helpers import LSE_TOL, SUM_TOL, dev, host, lse_err, norm_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def random_pattern(rng, M, N, n_rc, n_cc, p_keep=0.4):
    """Row clusters (with gaps) over [0, M), and per cluster sorted disjoint column ranges."""
    rc = np.sort(rng.choice(np.arange(1, M), 2 * n_rc - 1, replace=False))
    rc = np.concatenate([[0], rc, [M]])
    rows = np.array([[rc[2 * i], rc[2 * i + 1]] for i in range(n_rc)], dtype=np.int32)
    cc = np.concatenate([[0], np.sort(rng.choice(np.arange(1, N), n_cc - 1, replace=False)), [N]])
    ptr, cr = [0], []
    for i in range(n_rc):
        keep = np.nonzero(rng.uniform(size=n_cc) < p_keep)[0]
        cr.extend([cc[k], cc[k + 1]] for k in keep)
        ptr.append(len(cr))
    cr = np.array(cr, dtype=np.int32).reshape(-1, 2)
    return rows, np.array(ptr, dtype=np.int32), cr


def call(ctx, formula, reduction, x, y, b, pat, **kw):
    """kred_run_ranges (automatic column chunks unless col_blocks is given)."""
    import torch
    rows, ptr, cr = pat
    crt = dev(cr) if cr.size else torch.zeros((0, 2), dtype=torch.int32, device="cuda")
    return host(ctx.run_ranges(formula, reduction, dev(x), dev(y), None if b is None else dev(b),
                               dev(rows), dev(ptr), crt, **kw))


CHUNKS = [0, 1, 5]   # automatic, none, five column chunks per cluster


SUMS = [
    # formula, M, N, D, E, sigma, clusters (rows, cols)
    ("gauss", 3000, 4000, 3, 1, 0.1, (6, 10)),
    ("gauss", 5000, 3000, 2, 3, 0.2, (300, 40)),
    ("gauss", 800, 2500, 8, 20, 0.4, (5, 7)),
    ("laplace", 2000, 2000, 3, 4, 0.2, (9, 9)),
    ("sqdist", 1500, 1200, 16, 2, 1.0, (4, 6)),
]


@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("formula,M,N,D,E,sigma,cl", SUMS)
def test_ranges_sum(ctx, formula, M, N, D, E, sigma, cl, C):
    rng = np.random.default_rng(M + N + E)
    x = rng.uniform(0, 1, (M, D)).astype(np.float32)
    y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    pat = random_pattern(rng, M, N, *cl)
    out = call(ctx, formula, "sum", x, y, b, pat, sigma=sigma, col_blocks=C)
    ref, norm = oracle.ranges_reduce("sum", x, y, b, *pat, formula=formula, sigma=sigma)
    assert norm_err(out, ref, norm) <= SUM_TOL
    covered = np.zeros(M, bool)
    for r0, r1 in pat[0]:
        covered[r0:r1] = True
    assert (out[~covered] == 0).all()


def test_ranges_gradx(ctx):
    rng = np.random.default_rng(1)
    M, N = 4000, 3000
    x = rng.uniform(0, 1, (M, 3)).astype(np.float32); y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    pat = random_pattern(rng, M, N, 12, 15)
    for C in CHUNKS:
        out = call(ctx, "gauss_gradx", "sum", x, y, b, pat, sigma=0.1, col_blocks=C)
        ref, norm = oracle.ranges_reduce("gradx", x, y, b, *pat, sigma=0.1)
        assert norm_err(out, ref, norm) <= SUM_TOL
    ref, norm = oracle.ranges_reduce("gradx", x, y, b, *pat, sigma=0.1)
    assert norm_err(out, ref, norm) <= SUM_TOL


@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("formula,param", [("sinkhorn", 0.01), ("gauss", 0.1), ("laplace", 0.05)])
def test_ranges_lse(ctx, formula, param, C):
    rng = np.random.default_rng(2)
    M, N = 3000, 2500
    x = rng.uniform(0, 1, (M, 3)).astype(np.float32); y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
    g = (2.0 * rng.standard_normal((N, 1))).astype(np.float32)
    pat = random_pattern(rng, M, N, 10, 12)
    kw = dict(eps=param) if formula == "sinkhorn" else dict(sigma=param)
    out = call(ctx, formula, "lse", x, y, g, pat, col_blocks=C, **kw)
    okw = dict(eps=param) if formula == "sinkhorn" else dict(formula=formula, sigma=param)
    ref, m = oracle.ranges_reduce("lse", x, y, g, *pat, **okw)
    empty = np.isneginf(ref)
    assert (np.isneginf(out[empty, 0])).all()
    assert lse_err(out[~empty, 0], ref[~empty], m[~empty]) <= LSE_TOL


@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("red,K", [("argkmin", 5), ("kmin", 5), ("argkmin", 1)])
def test_ranges_knn_exact(ctx, red, K, C):
    rng = np.random.default_rng(3 + K)
    M, N, D = 2000, 3000, 4
    x = rng.integers(-3, 4, (M, D)).astype(np.float32); y = rng.integers(-3, 4, (N, D)).astype(np.float32)
    pat = random_pattern(rng, M, N, 8, 20, p_keep=0.15)   # some clusters get fewer than K columns
    out = call(ctx, "sqdist", red, x, y, None, pat, K=K, col_blocks=C)
    ref, _ = oracle.ranges_reduce(red, x, y, None, *pat, K=K)
    np.testing.assert_array_equal(out, ref.astype(out.dtype))


@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("red", ["min", "max", "argmin", "argmax"])
def test_ranges_extreme_exact(ctx, red, C):
    rng = np.random.default_rng(4)
    M, N = 1500, 2000
    x = rng.integers(-3, 4, (M, 3)).astype(np.float32); y = rng.integers(-3, 4, (N, 3)).astype(np.float32)
    b = rng.integers(-3, 4, (N, 2)).astype(np.float32)
    pat = random_pattern(rng, M, N, 7, 9)
    op = "max" if "max" in red else "min"
    for bb in (None, b):
        out = call(ctx, "sqdist", red, x, y, bb, pat, col_blocks=C)
        val, idx = oracle.ranges_reduce(op, x, y, bb, *pat, formula="sqdist")
        ref = idx.astype(np.int32) if red.startswith("arg") else val.astype(np.float32)
        np.testing.assert_array_equal(out, ref)


def test_ranges_clamped_and_empty_patterns(ctx):
    rng = np.random.default_rng(5)
    M, N = 600, 900
    x = rng.uniform(0, 1, (M, 3)).astype(np.float32); y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    # ranges reaching outside [0, M) x [0, N) are clamped; an inverted range is empty
    rows = np.array([[-50, 200], [400, 10 ** 6], [300, 250]], np.int32)
    ptr = np.array([0, 2, 3, 4], np.int32)
    cr = np.array([[-10, 100], [850, 5000], [100, 400], [0, 900]], np.int32)
    out = call(ctx, "gauss", "sum", x, y, b, (rows, ptr, cr), sigma=0.2)
    ref, norm = oracle.ranges_reduce("sum", x, y, b, rows, ptr, cr, formula="gauss", sigma=0.2)
    assert norm_err(out, ref, norm) <= SUM_TOL
    assert (out[200:400] == 0).all()
    # no clusters at all: every row holds the empty reduction
    empty = (np.zeros((0, 2), np.int32), np.zeros(1, np.int32), np.zeros((0, 2), np.int32))
    for C in CHUNKS:
        out = call(ctx, "gauss", "sum", x, y, b, empty, sigma=0.2, col_blocks=C)
        assert (out == 0).all()
        out = call(ctx, "sinkhorn", "lse", x, y, b, empty, eps=0.1, col_blocks=C)
        assert np.isneginf(out).all()


def test_ranges_full_pattern_matches_dense(ctx):
    # one cluster over everything reproduces kred_run (same kernels, no split;
    # the direct form on both sides, since dense sums this small otherwise take
    # the one-launch kernel)
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(6)
    M, N = 2500, 3500
    x = rng.uniform(0, 1, (M, 3)).astype(np.float32); y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
    b = rng.standard_normal((N, 2)).astype(np.float32)
    pat = (np.array([[0, M]], np.int32), np.array([0, 1], np.int32), np.array([[0, N]], np.int32))
    out = call(ctx, "gauss", "sum", x, y, b, pat, sigma=0.1, col_blocks=1, flags=kred.FLAG_DIRECT)
    dense = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=0.1, col_blocks=1,
                         flags=kred.FLAG_DIRECT))
    np.testing.assert_array_equal(out, dense)


FAST = [
    # formula, reduction, D, param, chunks
    ("gauss", "sum", 3, 0.05, 0), ("gauss", "sum", 2, 0.1, 1), ("gauss", "sum", 3, 0.05, 5),
    ("gauss_gradx", "sum", 3, 0.05, 0), ("gauss_gradx", "sum", 1, 0.1, 3),
    ("sinkhorn", "lse", 3, 0.01, 0), ("sinkhorn", "lse", 3, 0.01, 4), ("gauss", "lse", 2, 0.1, 0),
    ("gauss", "sum", 4, 0.05, 0), ("sinkhorn", "lse", 4, 0.01, 3),
]


@pytest.mark.parametrize("formula,reduction,D,param,C", FAST)
def test_ranges_fast_path(ctx, formula, reduction, D, param, C):
    # D <= 4 with KRED_FLAG_FAST: the matrix-core exponent kernel walks the
    # same pattern (ranges start and end anywhere, not on 16-column blocks)
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(D * 10 + C)
    M, N = 5000, 4000
    x = rng.uniform(0, 1, (M, D)).astype(np.float32); y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    pat = random_pattern(rng, M, N, 20, 30)
    kw = dict(eps=param) if formula == "sinkhorn" else dict(sigma=param)
    out = call(ctx, formula, reduction, x, y, b, pat, col_blocks=C, flags=kred.FLAG_FAST, **kw)
    if reduction == "lse":
        okw = dict(eps=param) if formula == "sinkhorn" else dict(formula=formula, sigma=param)
        ref, m = oracle.ranges_reduce("lse", x, y, b, *pat, **okw)
        empty = np.isneginf(ref)
        assert np.isneginf(out[empty, 0]).all()
        assert lse_err(out[~empty, 0], ref[~empty], m[~empty]) <= LSE_TOL
    elif formula == "gauss_gradx":
        ref, norm = oracle.ranges_reduce("gradx", x, y, b, *pat, sigma=param)
        assert norm_err(out, ref, norm) <= SUM_TOL
    else:
        ref, norm = oracle.ranges_reduce("sum", x, y, b, *pat, formula="gauss", sigma=param)
        assert norm_err(out, ref, norm) <= SUM_TOL


def test_ranges_fast_kernel_is_used(ctx):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(11)
    x = rng.uniform(0, 1, (3000, 3)).astype(np.float32); y = rng.uniform(0, 1, (3000, 3)).astype(np.float32)
    b = rng.standard_normal((3000, 1)).astype(np.float32)
    pat = random_pattern(rng, 3000, 3000, 6, 8)
    ctx.profile_collect()
    call(ctx, "gauss", "sum", x, y, b, pat, sigma=0.1, flags=kred.FLAG_FAST | kred.FLAG_PROFILE)
    n, ms, name = ctx.profile_collect()
    assert name == "fast_kernel"


@pytest.mark.parametrize("D", [3, 4])
@pytest.mark.parametrize("red", ["min", "argmin"])
def test_ranges_nearest_fast_path(ctx, red, D):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(13 + D)
    M, N = 4000, 5000
    x = rng.integers(-20, 21, (M, D)).astype(np.float32); y = rng.integers(-20, 21, (N, D)).astype(np.float32)
    pat = random_pattern(rng, M, N, 15, 25)
    for C in CHUNKS:
        out = call(ctx, "sqdist", red, x, y, None, pat, col_blocks=C, flags=kred.FLAG_FAST)
        val, idx = oracle.ranges_reduce("min", x, y, None, *pat, formula="sqdist")
        ref = idx.astype(np.int32) if red == "argmin" else val.astype(np.float32)
        np.testing.assert_array_equal(out, ref)


# ---------------------------------------------------------------- 16 < D <= 256
LARGE_SUMS = [
    # formula, M, N, D, E, sigma, clusters (rows, cols)
    ("gauss", 1500, 2000, 64, 16, 1.0, (6, 10)),
    ("gauss", 700, 1300, 128, 5, 1.2, (40, 25)),
    ("laplace", 900, 1100, 40, 3, 1.0, (5, 8)),
    ("sqdist", 600, 800, 33, 20, 1.0, (4, 6)),
    ("gauss", 300, 900, 256, 64, 1.0, (3, 5)),
]


@pytest.mark.parametrize("path", ["fp32", "split"])
@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("formula,M,N,D,E,sigma,cl", LARGE_SUMS)
def test_ranges_large_d_sum(ctx, formula, M, N, D, E, sigma, cl, C, path):
    # the matrix-core sums: fp32 products (KRED_FLAG_DIRECT) or split bf16 products
    # (KRED_FLAG_FAST); tiles start 16-aligned and mask the columns outside each range.
    # The Laplacian and squared-distance sums always take the fp64 contraction
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + N + E + D)
    x = (rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    pat = random_pattern(rng, M, N, *cl)
    fl = kred.FLAG_DIRECT if path == "fp32" else kred.FLAG_FAST
    ctx.profile_collect()
    out = call(ctx, formula, "sum", x, y, b, pat, sigma=sigma, col_blocks=C,
               flags=fl | kred.FLAG_PROFILE)
    want = ("mfma_f64_kernel" if formula in ("laplace", "sqdist")
            else "mfma_kernel" if path == "fp32" else "mfma_split_kernel")
    assert ctx.profile_collect()[2] == want
    ref, norm = oracle.ranges_reduce("sum", x, y, b, *pat, formula=formula, sigma=sigma)
    assert norm_err(out, ref, norm) <= SUM_TOL
    covered = np.zeros(M, bool)
    for r0, r1 in pat[0]:
        covered[r0:r1] = True
    assert (out[~covered] == 0).all()


@pytest.mark.parametrize("path", ["fp32", "exact"])
@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("red,K,D", [("argkmin", 10, 64), ("kmin", 5, 40), ("argkmin", 1, 128),
                                     ("argkmin", 16, 200), ("kmin", 64, 24)])
def test_ranges_large_d_knn_exact(ctx, red, K, D, C, path):
    # integer coordinates: the fp32 kernel and the exact bf16 kernel must both
    # match the oracle bit for bit, ties included
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(7 + K + D)
    M, N = 1200, 2500
    x = rng.integers(-4, 5, (M, D)).astype(np.float32); y = rng.integers(-4, 5, (N, D)).astype(np.float32)
    y[N // 2:N // 2 + N // 10] = y[:N // 10]
    pat = random_pattern(rng, M, N, 7, 18, p_keep=0.3)   # some clusters get fewer than K columns
    fl = kred.FLAG_DIRECT if path == "fp32" else kred.FLAG_FAST
    ctx.profile_collect()
    out = call(ctx, "sqdist", red, x, y, None, pat, K=K, col_blocks=C, flags=fl | kred.FLAG_PROFILE)
    assert ctx.profile_collect()[2] == ("mfma_kernel" if path == "fp32" else "knn_bf16_kernel")
    ref, _ = oracle.ranges_reduce(red, x, y, None, *pat, K=K)
    np.testing.assert_array_equal(out, ref.astype(out.dtype))


@pytest.mark.parametrize("red", ["min", "argmin"])
def test_ranges_large_d_nearest(ctx, red):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(12)
    M, N, D = 900, 1700, 48
    x = rng.integers(-4, 5, (M, D)).astype(np.float32); y = rng.integers(-4, 5, (N, D)).astype(np.float32)
    pat = random_pattern(rng, M, N, 9, 12)
    out = call(ctx, "sqdist", red, x, y, None, pat, flags=kred.FLAG_FAST)
    val, idx = oracle.ranges_reduce("min", x, y, None, *pat, formula="sqdist")
    ref = idx.astype(np.int32) if red == "argmin" else val.astype(np.float32)
    np.testing.assert_array_equal(out.reshape(ref.shape), ref)


def test_ranges_large_d_full_pattern_matches_dense(ctx):
    # one cluster holding every row and every column: same values as kred_run
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(13)
    M, N, D, E = 777, 1333, 96, 16
    x = (rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    pat = (np.array([[0, M]], np.int32), np.array([0, 1], np.int32), np.array([[0, N]], np.int32))
    for fl in (kred.FLAG_DIRECT, kred.FLAG_FAST):
        dense = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=1.0, col_blocks=1, flags=fl))
        sparse = call(ctx, "gauss", "sum", x, y, b, pat, sigma=1.0, col_blocks=1, flags=fl)
        np.testing.assert_array_equal(sparse, dense)


@pytest.mark.parametrize("C", CHUNKS)
@pytest.mark.parametrize("red,K", [("argkmin", 5), ("kmin", 10), ("argkmin", 16)])
def test_ranges_knn_fast_path(ctx, red, K, C):
    # D <= 3 with KRED_FLAG_FAST: the K-nearest lists on the matrix-core distance
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(40 + K)
    M, N, D = 2500, 3500, 3
    x = rng.integers(-9, 10, (M, D)).astype(np.float32); y = rng.integers(-9, 10, (N, D)).astype(np.float32)
    pat = random_pattern(rng, M, N, 9, 22, p_keep=0.2)   # some clusters get fewer than K columns
    ctx.profile_collect()
    out = call(ctx, "sqdist", red, x, y, None, pat, K=K, col_blocks=C, flags=kred.FLAG_FAST | kred.FLAG_PROFILE)
    assert ctx.profile_collect()[2] == "fast_kernel"
    ref, _ = oracle.ranges_reduce(red, x, y, None, *pat, K=K)
    np.testing.assert_array_equal(out, ref.astype(out.dtype))
