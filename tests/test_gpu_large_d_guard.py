"""GPU parity of the large-D expanded form's accuracy guard (16 < D <= 256).

The matrix-core kernels form T = fl(P + fl(nx + ny)) with P = sum_d 2 Y_d X_d
accumulated from zero and the centred coordinates and norms prepared in fp64;
their error in T is below (D + 10) 2^-24 L (fp32 products) or (D / 2 + 18)
2^-24 L (split bf16 products) with L = c (max |x - m|^2 + max |y - m|^2).
Above the budget (1.2e-4 in log2 units) the device routes the reduction to
the fp64 contraction; the Laplacian forms and the squared distance's sums and
extremes always take it.  These cases check which kernel ran (the profile
reports the device's choice) on both sides of each limit, data spread far
wider than the kernel width (where the fp32 expanded form would miss the
bar), adversarial data just inside the limits (far from the centre, close
pairs), and the oracle parity of every result; and the large-D k-NN values,
re-ranked by their direct-form distance.
"""
import numpy as np
import pytest

import oracle
from helpers import LSE_TOL, SUM_TOL, dev, grad_err_sigma, host, lse_err, norm_err

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
LOG2E = 1.4426950408889634


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def guard_L(x, y, c):
    """L of the guard: c (max |x - m|^2 + max |y - m|^2), m the mean of y's first 256 rows."""
    m = y[:256].astype(np.float64).mean(0)
    return c * (((x - m) ** 2).sum(1).max() + ((y - m) ** 2).sum(1).max())


def limit(D, split=False):
    """The largest L the fp32 (or split bf16) kernel takes at dimension D."""
    return 1.2e-4 / (((0.5 * D + 18) if split else (D + 10)) * U)


def expect_fp64(D, L, split=False):
    return L > limit(D, split)


def clustered(rng, n, D, ncl=6, far=3.0, near=0.05):
    """Points near a few centres spread far apart: close pairs matter, the box is wide."""
    centres = far * rng.standard_normal((ncl, D))
    lab = rng.integers(0, ncl, n)
    return (centres[lab] + near * rng.standard_normal((n, D))).astype(np.float32)


def _profiled(ctx, *args, **kw):
    from paper_2004_11127_amd import kred
    ctx.profile_collect()
    out = host(ctx.run(*args, flags=kw.pop("flags", 0) | kred.FLAG_PROFILE, **kw))
    return out, ctx.profile_collect()[2]


@pytest.mark.parametrize("D", [64, 128])
def test_verdict_cases_unit_variance(ctx, D):
    # unit-variance coordinates, eps = 0.01 and sigma = 0.02: the guard must
    # pick the fp64 contraction, and the results match the oracle.  Half of x
    # are points of y, whose self-pairs carry the sums (every other pair
    # underflows); the fp32 expanded form would be off by a factor of several
    rng = np.random.default_rng(D)
    M, N = 300, 800
    y = rng.standard_normal((N, D)).astype(np.float32)
    x = np.concatenate([y[N - M // 2:], rng.standard_normal((M - M // 2, D))]).astype(np.float32)
    g = rng.standard_normal((N, 1)).astype(np.float32)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    assert expect_fp64(D, guard_L(x, y, LOG2E / 0.01))
    out, name = _profiled(ctx, "sinkhorn", "lse", dev(x), dev(y), dev(g), eps=0.01)
    assert name == "mfma_f64_kernel"
    ref, m = oracle.sinkhorn_lse(x, y, g, 0.01)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL
    out, name = _profiled(ctx, "gauss", "sum", dev(x), dev(y), dev(b), sigma=0.02)
    assert name == "mfma_f64_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.02)
    assert norm_err(out, ref, norm) <= SUM_TOL


CLUSTER_CASES = [
    # formula, reduction, D, E, param (sigma or eps), col_blocks, flags
    ("gauss", "sum", 64, 1, 0.3, 0, 0),
    ("gauss", "sum", 128, 16, 0.3, 3, 0),
    ("gauss", "sum", 100, 3, 0.3, 0, 4),        # FLAG_FAST: the split kernel's place
    ("gauss", "sum", 256, 2, 0.4, 0, 0),
    ("sinkhorn", "lse", 64, 1, 0.2, 0, 0),
    ("sinkhorn", "lse", 200, 1, 0.2, 5, 0),
    ("gauss", "lse", 48, 1, 0.3, 0, 0),
    ("gauss", "max", 40, 3, 0.3, 0, 0),
    ("gauss_gradx", "sum", 64, 1, 0.3, 0, 0),
]


@pytest.mark.parametrize("formula,reduction,D,E,param,C,flags", CLUSTER_CASES)
def test_wide_clustered_data_takes_fp64(ctx, formula, reduction, D, E, param, C, flags):
    # clusters of radius about 0.05 sqrt(D) spread over about 3 sqrt(D): the
    # fp32 expanded form's bound is far above the budget (its error would be
    # about 1e-3 relative), the close pairs carry the sums
    rng = np.random.default_rng(D + E + C)
    M, N = 400, 1500
    y = clustered(rng, N, D)
    x = np.concatenate([y[:M // 2], clustered(rng, M - M // 2, D)])   # half of x in y
    b = rng.standard_normal((N, E)).astype(np.float32)
    kw = dict(eps=param) if formula == "sinkhorn" else dict(sigma=param)
    c = LOG2E / param if formula == "sinkhorn" else LOG2E / (2 * param * param)
    assert expect_fp64(D, guard_L(x, y, c)) and expect_fp64(D, guard_L(x, y, c), split=True)
    out, name = _profiled(ctx, formula, reduction, dev(x), dev(y), dev(b), col_blocks=C,
                          flags=flags, **kw)
    assert name == "mfma_f64_kernel", name
    if reduction == "lse":
        ref, m = (oracle.sinkhorn_lse(x, y, b, param) if formula == "sinkhorn"
                  else oracle.kernel_lse("gauss", x, y, b, param))
        assert lse_err(out[:, 0], ref, m) <= LSE_TOL
    elif reduction == "max":
        val, idx, scale = oracle.extreme("gauss", "max", x, y, b, param=param)
        assert (np.abs(out - val) <= 1e-4 * scale).all()
    elif formula == "gauss_gradx":
        ref, norm = oracle.gauss_gradx(x, y, b, param)
        assert norm_err(out[:, :1], ref[:, :1], norm[:, :1]) <= SUM_TOL
        assert grad_err_sigma(out, ref, norm, param) <= SUM_TOL
    else:
        ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=param)
        assert norm_err(out, ref, norm) <= SUM_TOL


@pytest.mark.parametrize("formula,reduction", [("laplace", "sum"), ("laplace", "lse"),
                                               ("sqdist", "sum"), ("laplace", "min")])
def test_sqrt_and_sqdist_forms_always_take_fp64(ctx, formula, reduction):
    # x a subset of y: distance-0 pairs, where sqrt of an absolute error e is sqrt(e)
    rng = np.random.default_rng(7)
    D, M, N = 32, 300, 1000
    y = (rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    x = y[:M].copy()
    b = rng.standard_normal((N, 1)).astype(np.float32)
    out, name = _profiled(ctx, formula, reduction, dev(x), dev(y), dev(b), sigma=0.2)
    assert name == "mfma_f64_kernel", name
    if reduction == "lse":
        ref, m = oracle.kernel_lse(formula, x, y, b, 0.2)
        assert lse_err(out[:, 0], ref, m) <= LSE_TOL
    elif reduction == "min":
        val, idx, scale = oracle.extreme(formula, "min", x, y, b, param=0.2)
        assert (np.abs(out - val) <= 1e-4 * scale).all()
    else:
        ref, norm = oracle.kernel_sum(formula, x, y, b, sigma=0.2)
        assert norm_err(out, ref, norm) <= SUM_TOL


@pytest.mark.parametrize("workload", ["c4", "gradx_d128"])
def test_workload_data_stays_on_fp32(ctx, workload):
    # N(0, I/128) at sigma = 1 (L about 2): inside the guard, the fp32 kernels run
    from paper_2004_11127_amd import inputs, kred
    w = inputs.highdim_gauss(M=2000, N=3000, D=128, E=16 if workload == "c4" else 1, sigma=1.0,
                             seed=0)
    assert not expect_fp64(128, guard_L(w.x, w.y, LOG2E / 2.0), split=True)
    formula = "gauss" if workload == "c4" else "gauss_gradx"
    out, name = _profiled(ctx, formula, "sum", dev(w.x), dev(w.y), dev(w.b), sigma=1.0,
                          flags=kred.FLAG_FAST)
    assert name == "mfma_split_kernel"
    if workload == "c4":
        ref, norm = oracle.kernel_sum("gauss", w.x, w.y, w.b, sigma=1.0)
        assert norm_err(out, ref, norm) <= SUM_TOL
    else:
        ref, norm = oracle.gauss_gradx(w.x, w.y, w.b, 1.0)
        assert norm_err(out, ref, norm) <= SUM_TOL


def test_lse_d64_data_stays_on_fp32(ctx):
    # the Sinkhorn workload's data (uniform / shifted uniform, D = 64, eps = 1):
    # L about 22, inside the fp32 kernel's limit (27.2)
    from paper_2004_11127_amd import inputs
    w = inputs.sinkhorn_lse(M=3000, N=3000, D=64, eps=1.0, seed=3)
    assert not expect_fp64(64, guard_L(w.x, w.y, LOG2E))
    g = w.b.reshape(-1, 1)
    out, name = _profiled(ctx, "sinkhorn", "lse", dev(w.x), dev(w.y), dev(g), eps=1.0)
    assert name == "mfma_kernel"
    ref, m = oracle.sinkhorn_lse(w.x, w.y, g, 1.0)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def two_clusters(rng, M, N, D, R=1.0, std=0.05):
    """y in two tight clusters at +-R along a random direction (the centre of y
    falls between them), x near points of y: every point about R from the
    centre, the informative pairs close."""
    u = rng.standard_normal(D); u /= np.linalg.norm(u)
    side = np.where(rng.uniform(size=N) < 0.5, -1.0, 1.0)
    y = side[:, None] * R * u + std * rng.standard_normal((N, D))
    x = y[rng.integers(0, N, M)] + 0.5 * std * rng.standard_normal((M, D))
    return x.astype(np.float32), y.astype(np.float32)


@pytest.mark.parametrize("D", [24, 64, 200])
@pytest.mark.parametrize("kind", ["sum_f32", "sum_split", "lse"])
def test_adversarial_data_just_inside_the_limit(ctx, D, kind):
    # c chosen so that L is 97% of the kernel's limit: the fp32 (or split)
    # kernel runs, on data where its rounding is largest (|x'|, |y'| at the
    # scale of sqrt(L) for every pair), and meets the bar
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(D + len(kind))
    M, N = 600, 2000
    x, y = two_clusters(rng, M, N, D, std=0.3 / np.sqrt(D))
    split = kind == "sum_split"
    c = 0.97 * limit(D, split) / guard_L(x, y, 1.0)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    if kind == "lse":
        eps = LOG2E / c
        out, name = _profiled(ctx, "sinkhorn", "lse", dev(x), dev(y), dev(b), eps=eps)
        assert name == "mfma_kernel"
        ref, m = oracle.sinkhorn_lse(x, y, b, eps)
        assert lse_err(out[:, 0], ref, m) <= LSE_TOL
    else:
        sigma = float(np.sqrt(LOG2E / (2 * c)))
        fl = kred.FLAG_FAST if split else kred.FLAG_DIRECT
        out, name = _profiled(ctx, "gauss", "sum", dev(x), dev(y), dev(b), sigma=sigma, flags=fl)
        assert name == ("mfma_split_kernel" if split else "mfma_kernel")
        ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=sigma)
        assert norm_err(out, ref, norm) <= SUM_TOL


@pytest.mark.parametrize("D", [20, 96, 256])
@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("side", [0.98, 1.02])
def test_guard_takes_the_side_of_the_limit(ctx, D, split, side):
    # the same data with c at 98% and 102% of the limit: fp32 (or split) below,
    # fp64 above, both at the bar
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(D)
    M, N = 300, 700
    x, y = two_clusters(rng, M, N, D, std=0.3 / np.sqrt(D))
    b = rng.standard_normal((N, 2)).astype(np.float32)
    c = side * limit(D, split) / guard_L(x, y, 1.0)
    sigma = float(np.sqrt(LOG2E / (2 * c)))
    fl = kred.FLAG_FAST if split else kred.FLAG_DIRECT
    out, name = _profiled(ctx, "gauss", "sum", dev(x), dev(y), dev(b), sigma=sigma, flags=fl)
    if side > 1:
        assert name == "mfma_f64_kernel"
    else:
        assert name == ("mfma_split_kernel" if split else "mfma_kernel")
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=sigma)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_block_sparse_fp64(ctx):
    # the fp64 variant with its own block-sparse workgroup map (one row block per wave at D = 128)
    from test_gpu_ranges import random_pattern
    rng = np.random.default_rng(11)
    D, M, N = 128, 900, 1400
    y = clustered(rng, N, D); x = clustered(rng, M, D)
    b = rng.standard_normal((N, 2)).astype(np.float32)
    rows, ptr, cr = random_pattern(rng, M, N, 9, 12)
    for C in (0, 1, 3):
        out = host(ctx.run_ranges("gauss", "sum", dev(x), dev(y), dev(b), dev(rows), dev(ptr),
                                  dev(cr), sigma=0.3, col_blocks=C))
        ref, norm = oracle.ranges_reduce("sum", x, y, b, rows, ptr, cr, formula="gauss", sigma=0.3)
        assert norm_err(out, ref, norm) <= SUM_TOL, C


@pytest.mark.parametrize("D,K,C", [(48, 5, 0), (100, 10, 3), (256, 1, 0)])
def test_large_d_knn_values_re_ranked(ctx, D, K, C):
    # real-valued points: the K-min values are the direct-form fp32 distances of
    # the returned points, and within the fp32 ranking bound of the true K smallest
    rng = np.random.default_rng(D + K)
    M, N = 500, 3000
    x = (3.0 + rng.standard_normal((M, D))).astype(np.float32)
    y = (3.0 + rng.standard_normal((N, D))).astype(np.float32)
    kd = host(ctx.run("sqdist", "kmin", dev(x), dev(y), None, K=K, col_blocks=C))
    idx = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=K, col_blocks=C))
    ridx, rdist = oracle.argkmin(x, y, K)
    # ranking by |y|^2 - 2 <x, y> in fp32: error below 2 (D + 2) 2^-24 (|x|^2 + |y|^2)
    span = (x.astype(np.float64) ** 2).sum(1).max() + (y.astype(np.float64) ** 2).sum(1).max()
    allow = 2 * 2 * (D + 2) * U * span + 8 * U * rdist
    assert (np.abs(kd.astype(np.float64) - rdist) <= allow).all()
    got = ((x[:, None, :].astype(np.float64) - y[idx].astype(np.float64)) ** 2).sum(-1)
    assert (np.abs(got - rdist) <= allow).all()
    # the values are the direct-form fp32 distances of the returned indices
    # (a sum of D non-negative terms: relative error below (D + 1) 2^-24)
    assert (np.abs(kd.astype(np.float64) - got) <= (D + 2) * U * got + 1e-30).all()


@pytest.mark.parametrize("D", [24, 40, 64, 100, 128])
@pytest.mark.parametrize("side", [0.97, 1.02])
def test_split_lse_guard_sides(ctx, D, side):
    # the Sinkhorn log-sum-exp on the split kernel (KRED_FLAG_FAST, D = 17..128):
    # at 97% of the split limit it runs there and meets the bar on data where
    # its rounding is largest; at 102% the fp64 contraction takes it
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(D + 7)
    M, N = 400, 1500
    x, y = two_clusters(rng, M, N, D, std=0.3 / np.sqrt(D))
    g = rng.standard_normal((N, 1)).astype(np.float32)
    c = side * limit(D, True) / guard_L(x, y, 1.0)
    eps = LOG2E / c
    out, name = _profiled(ctx, "sinkhorn", "lse", dev(x), dev(y), dev(g), eps=eps, flags=kred.FLAG_FAST)
    assert name == ("mfma_f64_kernel" if side > 1 else "mfma_split_kernel")
    ref, m = oracle.sinkhorn_lse(x, y, g, eps)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def test_lse_d64_data_on_the_split_kernel(ctx):
    # the lse_d64 workload's data with KRED_FLAG_FAST (as at its full size):
    # inside the split limit, on the split kernel, at the bar
    from paper_2004_11127_amd import inputs, kred
    w = inputs.sinkhorn_lse(M=3000, N=3000, D=64, eps=1.0, seed=3)
    assert not expect_fp64(64, guard_L(w.x, w.y, LOG2E), split=True)
    g = w.b.reshape(-1, 1)
    out, name = _profiled(ctx, "sinkhorn", "lse", dev(w.x), dev(w.y), dev(g), eps=1.0,
                          flags=kred.FLAG_FAST)
    assert name == "mfma_split_kernel"
    ref, m = oracle.sinkhorn_lse(w.x, w.y, g, 1.0)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL
