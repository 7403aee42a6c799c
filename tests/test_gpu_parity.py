"""GPU parity: libkred against the fp64 oracle, element by element, through the C ABI.

Small ragged shapes that span several row blocks, column tiles and a ragged
tail, every (formula, reduction) pair, forced column splits (second pass),
edge cases (M = 0, N = 0, single rows and columns), determinism and stream use.
"""
import numpy as np
import pytest

import oracle
from helpers import (LSE_TOL, SUM_TOL, dev, fast_L, fast_limit, fast_scale, host, lse_err,
                     norm_err, true_dists)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def _pts(rng, n, D, scale=1.0):
    return (rng.uniform(0.0, 1.0, (n, D)) * scale).astype(np.float32)


SUM_CASES = [
    # formula, M, N, D, E, sigma, col_blocks
    ("gauss", 1, 1, 3, 1, 0.3, 0),
    ("gauss", 7, 63, 3, 1, 0.3, 0),
    ("gauss", 65, 257, 3, 1, 0.2, 1),
    ("gauss", 1000, 4099, 3, 1, 0.1, 0),
    ("gauss", 4099, 1000, 3, 1, 0.1, 7),
    ("gauss", 2049, 1031, 1, 1, 0.05, 2),
    ("gauss", 513, 777, 2, 3, 0.1, 64),
    ("gauss", 300, 1500, 4, 16, 0.2, 0),
    ("gauss", 300, 1500, 5, 17, 0.3, 3),
    ("gauss", 129, 999, 8, 40, 0.4, 1),
    ("gauss", 257, 700, 16, 2, 0.6, 0),
    ("gauss", 100, 333, 9, 64, 0.5, 5),
    ("laplace", 1000, 4099, 3, 1, 0.1, 0),
    ("laplace", 77, 500, 7, 4, 0.3, 7),
    ("laplace", 3000, 200, 16, 1, 0.5, 1),
    ("sqdist", 1000, 4099, 3, 1, 1.0, 0),
    ("sqdist", 333, 1234, 12, 5, 1.0, 2),
    ("sqdist", 65, 64, 1, 16, 1.0, 64),
]


@pytest.mark.parametrize("formula,M,N,D,E,sigma,C", SUM_CASES)
def test_sum_parity(ctx, formula, M, N, D, E, sigma, C):
    rng = np.random.default_rng(M * 7 + N * 3 + D + E)
    x = _pts(rng, M, D); y = _pts(rng, N, D)
    b = rng.standard_normal((N, E)).astype(np.float32)
    out = host(ctx.run(formula, "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C))
    ref, norm = oracle.kernel_sum(formula, x, y, b, sigma=sigma)
    assert out.shape == (M, E)
    assert norm_err(out, ref, norm) <= SUM_TOL


GRADX_CASES = [
    (1, 1, 3, 0.3, 0), (7, 63, 3, 0.2, 0), (1000, 4099, 3, 0.1, 0), (4099, 1000, 3, 0.05, 7),
    (2049, 517, 1, 0.05, 2), (300, 999, 2, 0.1, 64), (257, 1200, 5, 0.3, 1), (129, 700, 16, 0.6, 3),
]


@pytest.mark.parametrize("M,N,D,sigma,C", GRADX_CASES)
def test_gradx_parity(ctx, M, N, D, sigma, C):
    rng = np.random.default_rng(M + 11 * N + D)
    x = _pts(rng, M, D); y = _pts(rng, N, D)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    out = host(ctx.run("gauss_gradx", "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C))
    ref, norm = oracle.gauss_gradx(x, y, b, sigma)
    assert out.shape == (M, 1 + D)
    assert norm_err(out, ref, norm) <= SUM_TOL


LSE_CASES = [
    (1, 1, 3, 0.1, 0), (7, 63, 3, 0.05, 0), (1000, 4099, 3, 0.01, 0), (4099, 1000, 3, 0.01, 7),
    (2049, 777, 1, 0.001, 2), (300, 1500, 2, 0.02, 64), (257, 999, 6, 0.1, 1), (65, 640, 16, 0.5, 3),
]


@pytest.mark.parametrize("M,N,D,eps,C", LSE_CASES)
def test_lse_parity(ctx, M, N, D, eps, C):
    rng = np.random.default_rng(M + 5 * N + D)
    x = _pts(rng, M, D); y = _pts(rng, N, D)
    y[:, 0] += 0.3
    g = rng.standard_normal((N, 1)).astype(np.float32)
    out = host(ctx.run("sinkhorn", "lse", dev(x), dev(y), dev(g), eps=eps, col_blocks=C))
    ref, m = oracle.sinkhorn_lse(x, y, g, eps)
    assert out.shape == (M, 1)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def test_lse_far_rows_and_large_offsets(ctx):
    # rows far from every column (all terms tiny) and a large shift of g: the
    # running maximum must keep every row finite and accurate
    rng = np.random.default_rng(3)
    x = _pts(rng, 500, 3, 4.0); y = _pts(rng, 2000, 3)
    g = (rng.standard_normal((2000, 1)) - 40.0).astype(np.float32)
    out = host(ctx.run("sinkhorn", "lse", dev(x), dev(y), dev(g), eps=0.05))
    ref, m = oracle.sinkhorn_lse(x, y, g, 0.05)
    assert np.all(np.isfinite(out))
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def _int_pts(rng, n, D, lo=-3, hi=3):
    return rng.integers(lo, hi + 1, (n, D)).astype(np.float32)


KNN_CASES = [
    # M, N, D, K, col_blocks
    (1, 1, 3, 1, 0), (7, 63, 3, 4, 0), (1000, 4099, 3, 10, 0), (4099, 1000, 2, 16, 7),
    (513, 2000, 8, 1, 2), (300, 999, 5, 32, 64), (129, 700, 16, 64, 3), (65, 64, 4, 64, 1),
    (2000, 3000, 3, 3, 0),
]


@pytest.mark.parametrize("M,N,D,K,C", KNN_CASES)
def test_argkmin_integer_bit_exact(ctx, M, N, D, K, C):
    # integer coordinates in a small box: many equal distances, exact in fp32
    rng = np.random.default_rng(M + 3 * N + D + K)
    x = _int_pts(rng, M, D); y = _int_pts(rng, N, D)
    out = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=K, col_blocks=C))
    ref, _ = oracle.argkmin(x, y, K)
    assert out.dtype == np.int32 and out.shape == (M, K)
    np.testing.assert_array_equal(out, ref)


def test_argkmin_float_coordinates(ctx):
    # non-integer data: fp32 rounding may reorder near-ties, so compare the
    # selected distances (fp64) with the oracle's and check validity
    rng = np.random.default_rng(17)
    x = _pts(rng, 700, 3); y = _pts(rng, 3001, 3)
    K = 10
    out = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=K))
    ref_idx, ref_d = oracle.argkmin(x, y, K)
    got_d = true_dists(x, y, np.arange(700), out)
    np.testing.assert_allclose(got_d, ref_d, rtol=1e-5, atol=1e-9)
    assert np.all((out >= 0) & (out < 3001))
    assert all(len(set(r)) == K for r in out.tolist())
    assert (out == ref_idx).mean() > 0.99


# ----------------------------------------------------------------- edge cases

def test_empty_m_is_noop(ctx):
    import torch
    x = torch.empty((0, 3), device="cuda"); y = dev(np.ones((5, 3), np.float32))
    b = dev(np.ones((5, 1), np.float32))
    out = ctx.run("gauss", "sum", x, y, b, sigma=1.0)
    assert out.shape == (0, 1)


def test_empty_n_gives_identity_of_the_reduction(ctx):
    import torch
    x = dev(np.ones((9, 3), np.float32)); y = torch.empty((0, 3), device="cuda")
    b = torch.empty((0, 2), device="cuda")
    out = host(ctx.run("gauss", "sum", x, y, b, sigma=1.0))
    assert out.shape == (9, 2) and not out.any()
    g = host(ctx.run("gauss_gradx", "sum", x, y, torch.empty((0, 1), device="cuda"), sigma=1.0))
    assert g.shape == (9, 4) and not g.any()
    l = host(ctx.run("sinkhorn", "lse", x, y, torch.empty((0, 1), device="cuda"), eps=1.0))
    assert np.all(np.isneginf(l))


def test_errors_raise_and_leave_output(ctx):
    import torch
    from paper_2004_11127_amd import kred
    x = dev(np.ones((4, 3), np.float32)); y = dev(np.ones((4, 3), np.float32))
    out = torch.full((4, 5), 7.0, device="cuda")
    with pytest.raises(kred.KredError):
        ctx.run("sqdist", "argkmin", x, y, None, K=5, out=torch.zeros((4, 5), dtype=torch.int32,
                                                                         device="cuda"))
    with pytest.raises(kred.KredError):
        ctx.run("gauss", "sum", x, y, dev(np.ones((4, 5), np.float32)), out=out, sigma=-1.0)
    assert torch.all(out == 7.0)


def test_deterministic_and_split_invariant(ctx):
    rng = np.random.default_rng(21)
    x = _pts(rng, 3000, 3); y = _pts(rng, 5000, 3)
    b = rng.standard_normal((5000, 1)).astype(np.float32)
    xd, yd, bd = dev(x), dev(y), dev(b)
    a1 = host(ctx.run("gauss", "sum", xd, yd, bd, sigma=0.1))
    a2 = host(ctx.run("gauss", "sum", xd, yd, bd, sigma=0.1))
    np.testing.assert_array_equal(a1, a2)
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.1)
    for C in (1, 3, 16, 200):
        aC = host(ctx.run("gauss", "sum", xd, yd, bd, sigma=0.1, col_blocks=C))
        assert norm_err(aC, ref, norm) <= SUM_TOL


def test_joint_permutation_of_columns(ctx):
    rng = np.random.default_rng(22)
    x = _pts(rng, 500, 3); y = _pts(rng, 2000, 3)
    b = rng.standard_normal((2000, 2)).astype(np.float32)
    p = rng.permutation(2000)
    a = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=0.2))
    ap = host(ctx.run("gauss", "sum", dev(x), dev(y[p]), dev(b[p]), sigma=0.2))
    _, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.2)
    assert norm_err(ap, a.astype(np.float64), norm) <= 2 * SUM_TOL


def test_runs_on_a_side_stream(ctx):
    import torch
    rng = np.random.default_rng(23)
    x = _pts(rng, 1000, 3); y = _pts(rng, 1000, 3)
    b = rng.standard_normal((1000, 1)).astype(np.float32)
    xd, yd, bd = dev(x), dev(y), dev(b)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        out = ctx.run("gauss", "sum", xd, yd, bd, sigma=0.1, stream=s)
    s.synchronize()
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.1)
    assert norm_err(host(out), ref, norm) <= SUM_TOL


def test_profile_collect_counts_launches(ctx):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(24)
    # 2^28+ pairs take the matrix-core exponent path; small problems the one-launch sum
    x = dev(_pts(rng, 20000, 3)); y = dev(_pts(rng, 16384, 3))
    b = dev(rng.standard_normal((16384, 1)).astype(np.float32))
    ctx.profile_collect()
    for _ in range(3):
        ctx.run("gauss", "sum", x, y, b, sigma=0.1, flags=kred.FLAG_PROFILE)
    n, ms, name = ctx.profile_collect()
    assert n == 3 and ms > 0 and name == "fast_kernel"
    for _ in range(2):
        ctx.run("gauss", "sum", x, y, b, sigma=0.1, flags=kred.FLAG_PROFILE | kred.FLAG_DIRECT)
    n, ms, name = ctx.profile_collect()
    assert n == 2 and ms > 0 and name == "sum_kernel"
    xs = dev(_pts(rng, 1000, 3))
    ctx.run("gauss", "sum", xs, y, b, sigma=0.1, flags=kred.FLAG_PROFILE)
    n, ms, name = ctx.profile_collect()
    assert n == 1 and name == "small_kernel"   # below 2^28 pairs: the one-launch sum


# ------------------------------------------------------- large D (matrix cores)

LARGE_SUM_CASES = [
    # formula, M, N, D, E, sigma, col_blocks
    ("gauss", 1, 1, 17, 1, 1.0, 0),
    ("gauss", 33, 47, 32, 16, 1.0, 0),
    ("gauss", 300, 1000, 128, 16, 1.0, 0),
    ("gauss", 1000, 777, 128, 16, 1.0, 3),
    ("gauss", 257, 1500, 64, 5, 0.7, 0),
    ("gauss", 129, 2001, 100, 17, 1.2, 2),
    ("gauss", 200, 900, 33, 40, 0.8, 1),
    ("gauss", 150, 640, 256, 64, 1.0, 5),
    ("gauss", 517, 333, 200, 1, 1.0, 64),
    ("laplace", 300, 1200, 64, 16, 1.0, 0),
    ("laplace", 77, 500, 128, 3, 2.0, 7),
    ("sqdist", 300, 1200, 64, 16, 1.0, 0),
    ("sqdist", 91, 450, 48, 2, 1.0, 3),
]


@pytest.mark.parametrize("formula,M,N,D,E,sigma,C", LARGE_SUM_CASES)
def test_large_d_sum_parity(ctx, formula, M, N, D, E, sigma, C):
    rng = np.random.default_rng(M * 3 + N + D * 7 + E)
    x = (rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    out = host(ctx.run(formula, "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C))
    ref, norm = oracle.kernel_sum(formula, x, y, b, sigma=sigma)
    assert out.shape == (M, E)
    assert norm_err(out, ref, norm) <= SUM_TOL


@pytest.mark.parametrize("formula,M,N,D,E,sigma,C", LARGE_SUM_CASES)
def test_large_d_sum_split_parity(ctx, formula, M, N, D, E, sigma, C):
    # KRED_FLAG_FAST: the contraction on the bf16 matrix cores with split
    # operands (6 partial products); fp32-level accuracy is expected, so the
    # error must stay within a few times the fp32 kernel's as well as the bar.
    # The Laplacian and squared-distance sums take the fp64 contraction instead
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M * 3 + N + D * 7 + E)
    x = (rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    ctx.profile_collect()
    out = host(ctx.run(formula, "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == ("mfma_f64_kernel" if formula in ("laplace", "sqdist")
                                        else "mfma_split_kernel")
    f32 = host(ctx.run(formula, "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C,
                       flags=kred.FLAG_DIRECT))
    ref, norm = oracle.kernel_sum(formula, x, y, b, sigma=sigma)
    e_split, e_f32 = norm_err(out, ref, norm), norm_err(f32, ref, norm)
    print("split %.3g  fp32 %.3g" % (e_split, e_f32))
    assert e_split <= SUM_TOL
    assert e_split <= max(4 * e_f32, 2e-6)


LARGE_KNN_CASES = [
    # M, N, D, K, col_blocks
    (1, 1, 17, 1, 0), (65, 300, 32, 10, 0), (300, 2000, 64, 10, 0), (1000, 1500, 64, 10, 5),
    (129, 777, 128, 16, 0), (100, 900, 200, 4, 2), (70, 640, 64, 64, 1), (513, 1001, 40, 1, 3),
    (64, 64, 64, 64, 0),
]


@pytest.mark.parametrize("M,N,D,K,C", LARGE_KNN_CASES)
def test_large_d_argkmin_integer_bit_exact(ctx, M, N, D, K, C):
    rng = np.random.default_rng(M + 3 * N + D + K)
    x = _int_pts(rng, M, D, -8, 8); y = _int_pts(rng, N, D, -8, 8)
    # duplicate some columns to force exact ties
    y[N // 2:N // 2 + N // 8] = y[:N // 8]
    out = host(ctx.run("sqdist", "argkmin", dev(x), dev(y), None, K=K, col_blocks=C))
    ref, _ = oracle.argkmin(x, y, K)
    np.testing.assert_array_equal(out, ref)


def test_large_d_unsupported_pairs_raise(ctx):
    # every valid pair is served at D > 16; a pair outside the table still fails
    from paper_2004_11127_amd import kred
    x = dev(np.ones((4, 32), np.float32)); y = dev(np.ones((4, 32), np.float32))
    with pytest.raises(kred.KredError) as e:
        ctx.run("sqdist", "lse", x, y, dev(np.ones((4, 1), np.float32)))
    assert e.value.status == 2


# ------------------------------------------- small-D matrix-core exponent path

FAST_CASES = [
    # formula, reduction, M, N, D, param, col_blocks
    ("gauss", "sum", 1, 1, 3, 0.3, 0),
    ("gauss", "sum", 7, 5, 3, 0.3, 0),
    ("gauss", "sum", 300, 17, 2, 0.2, 0),
    ("gauss", "sum", 1000, 4099, 3, 0.05, 0),
    ("gauss", "sum", 4099, 1000, 1, 0.02, 3),
    ("gauss", "sum", 2000, 3001, 3, 0.1, 16),
    ("gauss_gradx", "sum", 1, 1, 3, 0.3, 0),
    ("gauss_gradx", "sum", 1000, 4099, 3, 0.05, 0),
    ("gauss_gradx", "sum", 2049, 517, 2, 0.05, 2),
    ("gauss_gradx", "sum", 333, 2050, 1, 0.1, 7),
    ("sinkhorn", "lse", 1, 1, 3, 0.1, 0),
    ("sinkhorn", "lse", 9, 5, 3, 0.05, 0),
    ("sinkhorn", "lse", 1000, 4099, 3, 0.01, 0),
    ("sinkhorn", "lse", 4099, 1000, 2, 0.002, 3),
    ("sinkhorn", "lse", 700, 2001, 1, 0.01, 16),
    # four coordinates: six products per coordinate; the matrix-core path takes
    # c R^2 <= 128 (sigma = 0.1 and eps = 0.02 here), the direct form the rest
    ("gauss", "sum", 1000, 4099, 4, 0.1, 0),
    ("sinkhorn", "lse", 1000, 4099, 4, 0.02, 3),
    ("gauss", "sum", 1000, 4099, 4, 0.05, 0),
    ("gauss", "sum", 2000, 3001, 4, 0.1, 16),
    ("sinkhorn", "lse", 1000, 4099, 4, 0.01, 0),
    ("sinkhorn", "lse", 4099, 1000, 4, 0.002, 3),
    ("gauss_gradx", "sum", 1000, 4099, 4, 0.05, 0),   # the direct form (no fast gradient at D = 4)
]


_DIRECT = {"gauss": "sum_kernel", "gauss_gradx": "gradx_kernel", "sinkhorn": "lse_kernel"}


def _fast_case(ctx, formula, reduction, M, N, D, param, C, flags, scale=1.0):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + 17 * N + D)
    x = _pts(rng, M, D, scale); y = _pts(rng, N, D, scale)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    kw = dict(sigma=param) if reduction == "sum" else dict(eps=param)
    ctx.profile_collect()
    out = host(ctx.run(formula, reduction, dev(x), dev(y), dev(b), col_blocks=C,
                       flags=flags | kred.FLAG_PROFILE, **kw))
    # the kernel the device chose: the matrix-core exponent when FLAG_FAST, the
    # pair has one (the fused gradient up to D = 3) and c R^2 is inside the guard
    name = ctx.profile_collect()[2]
    has_fast = D <= 3 or formula != "gauss_gradx"
    inside = fast_L(x, y, fast_scale(formula, reduction, param)) <= fast_limit(D, False)
    want_fast = bool(flags & kred.FLAG_FAST) and has_fast and inside
    assert name == ("fast_kernel" if want_fast else _DIRECT[formula]), name
    if formula == "gauss":
        ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=param)
        err = norm_err(out, ref, norm)
        return err <= SUM_TOL, err
    if formula == "gauss_gradx":
        ref, norm = oracle.gauss_gradx(x, y, b, param)
        err = norm_err(out, ref, norm)
        return err <= SUM_TOL, err
    ref, m = oracle.sinkhorn_lse(x, y, b, param)
    err = lse_err(out[:, 0], ref, m)
    return err <= LSE_TOL, err


@pytest.mark.parametrize("formula,reduction,M,N,D,param,C", FAST_CASES)
def test_fast_path_parity(ctx, formula, reduction, M, N, D, param, C):
    from paper_2004_11127_amd import kred
    ok, err = _fast_case(ctx, formula, reduction, M, N, D, param, C, flags=kred.FLAG_FAST)
    assert ok, err


@pytest.mark.parametrize("formula,reduction,M,N,D,param,C", FAST_CASES[3:6] + FAST_CASES[7:9] + FAST_CASES[12:14])
def test_direct_flag_parity(ctx, formula, reduction, M, N, D, param, C):
    from paper_2004_11127_amd import kred
    ok, err = _fast_case(ctx, formula, reduction, M, N, D, param, C, flags=kred.FLAG_DIRECT)
    assert ok, err


@pytest.mark.parametrize("formula,reduction,param", [("gauss", "sum", 0.01), ("gauss_gradx", "sum", 0.01),
                                                     ("sinkhorn", "lse", 0.1)])
def test_fast_path_falls_back_on_wide_data(ctx, formula, reduction, param):
    # points spread over [0, 20]^3 with a narrow kernel: c R^2 is above the fast
    # path's limit (4300 for the log-sum-exp case, far more for the Gaussians),
    # so the direct-form kernels must produce the result
    from paper_2004_11127_amd import kred
    ok, err = _fast_case(ctx, formula, reduction, 500, 3000, 3, param, 0, flags=kred.FLAG_FAST,
                         scale=20.0)
    assert ok, err


@pytest.mark.parametrize("path", ["fast", "direct"])
@pytest.mark.parametrize("profile", ["rising", "falling", "spread"])
def test_lse_running_maximum(ctx, path, profile):
    # g_j chosen so the row maximum of s_ij = g_j - |x_i - y_j|^2 / eps moves by
    # far more than the rescale threshold inside a column range: "rising" puts
    # a new maximum in almost every tile (and inside tiles), "falling" puts it
    # in the first tile, "spread" scatters large values at random
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(5)
    M, N, eps = 777, 5000, 0.05
    x = _pts(rng, M, 3); y = _pts(rng, N, 3)
    ramp = np.linspace(0.0, 600.0, N)
    g = {"rising": ramp, "falling": ramp[::-1].copy(),
         "spread": 80.0 * rng.standard_normal(N)}[profile]
    g = g.astype(np.float32).reshape(N, 1)
    flags = kred.FLAG_FAST if path == "fast" else kred.FLAG_DIRECT
    for C in (0, 3):
        out = host(ctx.run("sinkhorn", "lse", dev(x), dev(y), dev(g), eps=eps, col_blocks=C,
                           flags=flags))
        ref, m = oracle.sinkhorn_lse(x, y, g, eps)
        err = lse_err(out[:, 0], ref, m)
        assert err <= LSE_TOL, (C, err)


def test_fast_path_deterministic(ctx):
    from paper_2004_11127_amd import kred
    F = kred.FLAG_FAST
    rng = np.random.default_rng(31)
    x = dev(_pts(rng, 3000, 3)); y = dev(_pts(rng, 5000, 3))
    b = dev(rng.standard_normal((5000, 1)).astype(np.float32))
    for f in ("gauss", "gauss_gradx"):
        a1 = host(ctx.run(f, "sum", x, y, b, sigma=0.05, flags=F))
        a2 = host(ctx.run(f, "sum", x, y, b, sigma=0.05, flags=F))
        np.testing.assert_array_equal(a1, a2)
    l1 = host(ctx.run("sinkhorn", "lse", x, y, b, eps=0.01, flags=F))
    l2 = host(ctx.run("sinkhorn", "lse", x, y, b, eps=0.01, flags=F))
    np.testing.assert_array_equal(l1, l2)


@pytest.mark.parametrize("formula,E", [("gauss", 1), ("laplace", 3), ("sqdist", 16)])
def test_direct_sum_both_row_counts(ctx, formula, E):
    # the direct sums run 2 rows per thread when the default grid would leave
    # CUs idle (small M) and their default row count otherwise; both must agree
    # with the oracle (sampled rows at the larger size)
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(31 + E)
    for M, N in ((3000, 4000), (60000, 20000)):
        x = _pts(rng, M, 3); y = _pts(rng, N, 3)
        b = rng.standard_normal((N, E)).astype(np.float32)
        out = host(ctx.run(formula, "sum", dev(x), dev(y), dev(b), sigma=0.1, flags=kred.FLAG_DIRECT))
        rows = np.sort(rng.choice(M, 300, replace=False))
        ref, norm = oracle.kernel_sum(formula, x, y, b, sigma=0.1, rows=rows)
        assert norm_err(out[rows], ref, norm) <= SUM_TOL


@pytest.mark.parametrize("M,N,D,E,sigma,C", [(1000, 4099, 3, 3, 0.05, 0), (2049, 777, 2, 2, 0.1, 5),
                                             (700, 2001, 4, 4, 0.08, 0), (1, 1, 3, 3, 0.3, 0),
                                             (3000, 2500, 1, 4, 0.02, 16)])
def test_fast_path_vector_signal(ctx, M, N, D, E, sigma, C):
    # Gaussian sums with 2 <= E <= 4 signal columns on the matrix-core exponent
    # path: the gradient's four accumulators carry b's columns
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(M + N + D + E)
    x = _pts(rng, M, D, 1.0); y = _pts(rng, N, D, 1.0)
    b = rng.standard_normal((N, E)).astype(np.float32)
    ctx.profile_collect()
    out = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=sigma, col_blocks=C,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == "fast_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=sigma)
    assert out.shape == (M, E)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_fast_path_vector_signal_ranges(ctx):
    from paper_2004_11127_amd import kred
    from test_gpu_ranges import random_pattern
    rng = np.random.default_rng(77)
    M, N = 3000, 3500
    x = _pts(rng, M, 3, 1.0); y = _pts(rng, N, 3, 1.0)
    b = rng.standard_normal((N, 3)).astype(np.float32)
    rows, ptr, cr = random_pattern(rng, M, N, 12, 20)
    for C in (0, 1, 4):
        out = host(ctx.run_ranges("gauss", "sum", dev(x), dev(y), dev(b), dev(rows), dev(ptr),
                                  dev(cr), sigma=0.05, col_blocks=C, flags=kred.FLAG_FAST))
        ref, norm = oracle.ranges_reduce("sum", x, y, b, rows, ptr, cr, formula="gauss", sigma=0.05)
        assert norm_err(out, ref, norm) <= SUM_TOL, C
