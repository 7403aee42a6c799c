"""Pins for the fp64 oracle, checked against what the mathematics fixes (CPU only).

The paper prints no worked numeric example, so the oracle is pinned by
hand-derived two-point values (tests/golden/hand_values.json), closed forms
that hold at any size (separable sums on Cartesian lattices, sigma -> infinity
limits, the expanded squared-distance identity), invariants (linearity,
translation and joint-permutation invariance, log-sum-exp shift), finite
differences for the gradient, and brute-force sorting for arg-K-min.  Each
check is chosen so that a plausible slip in the oracle (a dropped term, a
wrong sign, scale or index, a transposed operand, a wrong tie-break) fails.
"""
import json
import math
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_values.json")


@pytest.fixture(scope="module")
def hv():
    with open(GOLDEN) as f:
        return json.load(f)


def _a(v):
    return np.asarray(v, dtype=np.float64)


# ---------------------------------------------------------------- hand values

def test_golden_file_matches_its_closed_forms(hv):
    # The stored numbers are the closed forms written in each entry.
    assert hv["gauss_two_point"]["value"] == pytest.approx(1 + 2 * math.exp(-0.5), rel=1e-15)
    assert hv["gauss_two_point_scaled"]["value"] == pytest.approx(3 - math.exp(-2), rel=1e-15)
    assert hv["laplace_two_point"]["value"] == pytest.approx(1 + 2 * math.exp(-1), rel=1e-15)
    assert hv["lse_two_point"]["value"] == pytest.approx(math.log(2), rel=1e-15)
    assert hv["vjp_two_point"]["value"] == pytest.approx([5 * math.exp(-0.5), -6 * math.exp(-2)],
                                                         rel=1e-15)


@pytest.mark.parametrize("key,formula", [("gauss_two_point", "gauss"),
                                         ("gauss_two_point_scaled", "gauss"),
                                         ("laplace_two_point", "laplace"),
                                         ("sqdist_two_point", "sqdist")])
def test_sum_hand_values(oracle_mod, hv, key, formula):
    c = hv[key]
    a, n = oracle_mod.kernel_sum(formula, _a(c["x"]), _a(c["y"]), _a(c["b"]), sigma=c["sigma"])
    assert a[0, 0] == pytest.approx(c["value"], rel=1e-14, abs=1e-14)


def test_gradx_hand_value(oracle_mod, hv):
    c = hv["gradx_one_point"]
    out, norm = oracle_mod.gauss_gradx(_a(c["x"]), _a(c["y"]), _a(c["b"]), c["sigma"])
    np.testing.assert_allclose(out[0], c["value"], rtol=1e-14, atol=1e-15)


def test_lse_hand_value(oracle_mod, hv):
    c = hv["lse_two_point"]
    a, m = oracle_mod.sinkhorn_lse(_a(c["x"]), _a(c["y"]), _a(c["g"]), c["eps"])
    assert a[0] == pytest.approx(c["value"], rel=1e-14)
    assert m[0] == pytest.approx(0.0, abs=1e-15)


def test_argkmin_hand_value(oracle_mod, hv):
    c = hv["argkmin_small"]
    idx, dist = oracle_mod.argkmin(_a(c["x"]), _a(c["y"]), c["K"])
    assert idx[0].tolist() == c["value"]
    np.testing.assert_array_equal(dist[0], [0.0, 1.0, 1.0, 1.0])


# ---------------------------------------------------------- Gaussian closed forms

def _lattice(axes):
    g = np.meshgrid(*axes, indexing="ij")
    return np.stack([t.ravel() for t in g], axis=1)


@pytest.mark.parametrize("sigma", [0.07, 0.3, 1.7])
def test_gauss_separable_lattice(oracle_mod, sigma):
    # With b = 1 and y on a Cartesian lattice G1 x G2 x G3, Eq. (1) factorises:
    # a(x) = prod_d sum_{t in G_d} exp(-(x_d - t)^2 / (2 sigma^2)).
    # Axes of different lengths and spacings catch swapped coordinates.
    axes = [np.linspace(-0.3, 0.9, 5), np.linspace(0.1, 0.4, 3), np.array([-1.0, 0.0, 0.5, 2.0])]
    y = _lattice(axes)
    rng = np.random.default_rng(1)
    x = rng.uniform(-0.5, 1.0, (17, 3))
    b = np.ones((y.shape[0], 1))
    a, n = oracle_mod.kernel_sum("gauss", x, y, b, sigma=sigma)
    want = np.ones(x.shape[0])
    for d in range(3):
        want *= np.exp(-(x[:, d:d + 1] - axes[d][None, :]) ** 2 / (2 * sigma ** 2)).sum(axis=1)
    np.testing.assert_allclose(a[:, 0], want, rtol=1e-13)
    np.testing.assert_allclose(n[:, 0], want, rtol=1e-13)  # all terms positive


def test_gauss_separable_lattice_high_dim(oracle_mod):
    # Same identity in D = 6 with a two-point axis per dimension (64 lattice points).
    axes = [np.array([0.0, 0.1 * (d + 1)]) for d in range(6)]
    y = _lattice(axes)
    x = np.random.default_rng(2).normal(size=(5, 6)) * 0.2
    a, _ = oracle_mod.kernel_sum("gauss", x, y, np.ones((64, 1)), sigma=0.25)
    want = np.ones(5)
    for d in range(6):
        want *= np.exp(-(x[:, d:d + 1] - axes[d][None, :]) ** 2 / (2 * 0.25 ** 2)).sum(axis=1)
    np.testing.assert_allclose(a[:, 0], want, rtol=1e-13)


@pytest.mark.parametrize("formula", ["gauss", "laplace"])
def test_sigma_to_infinity_gives_sum_of_b(oracle_mod, formula):
    rng = np.random.default_rng(3)
    x = rng.uniform(0, 1, (9, 3)); y = rng.uniform(0, 1, (31, 3)); b = rng.normal(size=(31, 2))
    a, n = oracle_mod.kernel_sum(formula, x, y, b, sigma=1e9)
    np.testing.assert_allclose(a, np.broadcast_to(b.sum(axis=0), a.shape), rtol=1e-7, atol=1e-8)
    np.testing.assert_allclose(n, np.broadcast_to(np.abs(b).sum(axis=0), n.shape), rtol=1e-7)


def test_linearity_translation_permutation(oracle_mod):
    rng = np.random.default_rng(4)
    x = rng.uniform(0, 1, (13, 3)); y = rng.uniform(0, 1, (40, 3))
    b1 = rng.normal(size=(40, 3)); b2 = rng.normal(size=(40, 3))
    a1, _ = oracle_mod.kernel_sum("gauss", x, y, b1, sigma=0.2)
    a2, _ = oracle_mod.kernel_sum("gauss", x, y, b2, sigma=0.2)
    a12, _ = oracle_mod.kernel_sum("gauss", x, y, 2.0 * b1 - 3.0 * b2, sigma=0.2)
    np.testing.assert_allclose(a12, 2 * a1 - 3 * a2, rtol=1e-12, atol=1e-12)
    t = np.array([[5.0, -2.0, 0.25]])
    at, _ = oracle_mod.kernel_sum("gauss", x + t, y + t, b1, sigma=0.2)
    np.testing.assert_allclose(at, a1, rtol=1e-10, atol=1e-12)
    p = rng.permutation(40)
    ap, _ = oracle_mod.kernel_sum("gauss", x, y[p], b1[p], sigma=0.2)
    np.testing.assert_allclose(ap, a1, rtol=1e-12, atol=1e-13)


def test_rows_subset_matches_full(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.uniform(0, 1, (50, 3)); y = rng.uniform(0, 1, (60, 3)); b = rng.normal(size=(60, 1))
    full, _ = oracle_mod.kernel_sum("gauss", x, y, b, sigma=0.3)
    rows = np.array([0, 7, 49, 23])
    sub, _ = oracle_mod.kernel_sum("gauss", x, y, b, sigma=0.3, rows=rows)
    np.testing.assert_array_equal(sub, full[rows])


def test_empty_inputs(oracle_mod):
    x = np.zeros((3, 2)); y = np.zeros((0, 2)); b = np.zeros((0, 4))
    a, n = oracle_mod.kernel_sum("gauss", x, y, b, sigma=1.0)
    assert a.shape == (3, 4) and not a.any() and not n.any()
    l, _ = oracle_mod.sinkhorn_lse(x, y, np.zeros((0, 1)), 1.0)
    assert np.all(np.isneginf(l))


# ------------------------------------------------------------------ Laplace, SqDist

def test_laplace_two_points_on_axis(oracle_mod):
    # |x - y| = 2 and 0.5 on an axis: 1*exp(-2/0.5)... closed form per term.
    x = _a([[1.0, 1.0]]); y = _a([[3.0, 1.0], [1.0, 0.5]]); b = _a([[1.0], [-4.0]])
    a, n = oracle_mod.kernel_sum("laplace", x, y, b, sigma=0.5)
    assert a[0, 0] == pytest.approx(math.exp(-4.0) - 4.0 * math.exp(-1.0), rel=1e-14)
    assert n[0, 0] == pytest.approx(math.exp(-4.0) + 4.0 * math.exp(-1.0), rel=1e-14)


def test_sqdist_sum_expanded_identity(oracle_mod):
    # sum_j |x_i - y_j|^2 b_j = |x_i|^2 sum_j b_j - 2 <x_i, sum_j b_j y_j> + sum_j b_j |y_j|^2
    rng = np.random.default_rng(6)
    x = rng.normal(size=(11, 5)); y = rng.normal(size=(37, 5)); b = rng.normal(size=(37, 2))
    a, _ = oracle_mod.kernel_sum("sqdist", x, y, b)
    want = (np.sum(x * x, 1)[:, None] * b.sum(0)[None, :] - 2 * x @ (y.T @ b)
            + (np.sum(y * y, 1)[:, None] * b).sum(0)[None, :])
    np.testing.assert_allclose(a, want, rtol=1e-11, atol=1e-11)


# ------------------------------------------------------------------------ gradient

def test_gradx_column0_is_gauss_sum(oracle_mod):
    rng = np.random.default_rng(7)
    x = rng.uniform(0, 1, (8, 3)); y = rng.uniform(0, 1, (25, 3)); b = rng.normal(size=(25, 1))
    out, norm = oracle_mod.gauss_gradx(x, y, b, 0.3)
    a, n = oracle_mod.kernel_sum("gauss", x, y, b, sigma=0.3)
    np.testing.assert_allclose(out[:, 0], a[:, 0], rtol=1e-14)
    np.testing.assert_allclose(norm[:, 0], n[:, 0], rtol=1e-14)


@pytest.mark.parametrize("sigma,D", [(0.3, 3), (0.05, 3), (1.1, 5)])
def test_gradx_matches_finite_differences(oracle_mod, sigma, D):
    # g_ik = d a_i / d x_ik: central differences of the oracle's own a_i, in fp64.
    rng = np.random.default_rng(8)
    x = rng.uniform(0, 1, (6, D)) * (4 * sigma); y = rng.uniform(0, 1, (30, D)) * (4 * sigma)
    b = rng.normal(size=(30, 1))
    out, norm = oracle_mod.gauss_gradx(x, y, b, sigma)
    h = 1e-5 * sigma
    for k in range(D):
        xp = x.copy(); xp[:, k] += h
        xm = x.copy(); xm[:, k] -= h
        ap, _ = oracle_mod.kernel_sum("gauss", xp, y, b, sigma=sigma)
        am, _ = oracle_mod.kernel_sum("gauss", xm, y, b, sigma=sigma)
        fd = (ap[:, 0] - am[:, 0]) / (2 * h)
        np.testing.assert_allclose(out[:, 1 + k], fd, rtol=1e-6, atol=1e-7 * norm[:, 1 + k].max())


def test_vjp_hand_value(oracle_mod, hv):
    c = hv["vjp_two_point"]
    g, norm = oracle_mod.gauss_vjp(_a(c["x"]), _a(c["y"]), _a(c["b"]), _a(c["e"]), c["sigma"])
    np.testing.assert_allclose(g[0], c["value"], rtol=1e-14, atol=1e-15)


def _loss(oracle_mod, x, y, b, e, sigma):
    # L = sum_i <e_i, a_i> with a from the oracle's Gaussian sum
    a, _ = oracle_mod.kernel_sum("gauss", x, y, b, sigma=sigma)
    return float((a * e).sum())


@pytest.mark.parametrize("sigma,D,E", [(0.3, 3, 1), (0.2, 2, 4), (1.1, 5, 3)])
def test_vjp_matches_finite_differences(oracle_mod, sigma, D, E):
    # x-gradient, y-gradient (the same routine with the roles exchanged) and
    # b-gradient (the Gaussian sum with x and y exchanged) of L = sum_i <e_i, a_i>,
    # against central differences of L in fp64.
    rng = np.random.default_rng(9 + D + E)
    M, N = 5, 23
    x = rng.uniform(0, 1, (M, D)) * (4 * sigma); y = rng.uniform(0, 1, (N, D)) * (4 * sigma)
    b = rng.normal(size=(N, E)); e = rng.normal(size=(M, E))
    gx, nx = oracle_mod.gauss_vjp(x, y, b, e, sigma)
    gy, ny = oracle_mod.gauss_vjp(y, x, e, b, sigma)
    gb, _ = oracle_mod.kernel_sum("gauss", y, x, e, sigma=sigma)
    h = 1e-5 * sigma
    for (var, grad, scale) in (("x", gx, nx.max()), ("y", gy, ny.max())):
        base = x if var == "x" else y
        for i in range(base.shape[0]):
            for k in range(D):
                p = base.copy(); p[i, k] += h
                m = base.copy(); m[i, k] -= h
                if var == "x":
                    fd = (_loss(oracle_mod, p, y, b, e, sigma) - _loss(oracle_mod, m, y, b, e, sigma)) / (2 * h)
                else:
                    fd = (_loss(oracle_mod, x, p, b, e, sigma) - _loss(oracle_mod, x, m, b, e, sigma)) / (2 * h)
                assert grad[i, k] == pytest.approx(fd, rel=1e-6, abs=1e-7 * scale)
    for j in range(N):
        for c in range(E):
            p = b.copy(); p[j, c] += 1.0
            fd = _loss(oracle_mod, x, y, p, e, sigma) - _loss(oracle_mod, x, y, b, e, sigma)   # linear in b
            assert gb[j, c] == pytest.approx(fd, rel=1e-10, abs=1e-12)


def test_vjp_unit_cotangent_is_gradx(oracle_mod):
    # E = 1 and e = 1: the product is the x-gradient the fused routine returns
    rng = np.random.default_rng(10)
    x = rng.uniform(0, 1, (9, 3)); y = rng.uniform(0, 1, (31, 3)); b = rng.normal(size=(31, 1))
    g, n = oracle_mod.gauss_vjp(x, y, b, np.ones((9, 1)), 0.25)
    out, norm = oracle_mod.gauss_gradx(x, y, b, 0.25)
    np.testing.assert_allclose(g, out[:, 1:], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(n, norm[:, 1:], rtol=1e-13)


def test_vjp_linear_in_cotangent_and_signal(oracle_mod):
    rng = np.random.default_rng(11)
    x = rng.uniform(0, 1, (7, 2)); y = rng.uniform(0, 1, (19, 2))
    b = rng.normal(size=(19, 3)); e1 = rng.normal(size=(7, 3)); e2 = rng.normal(size=(7, 3))
    g1, _ = oracle_mod.gauss_vjp(x, y, b, e1, 0.4)
    g2, _ = oracle_mod.gauss_vjp(x, y, b, e2, 0.4)
    g12, _ = oracle_mod.gauss_vjp(x, y, b, e1 - 2 * e2, 0.4)
    np.testing.assert_allclose(g12, g1 - 2 * g2, rtol=1e-12, atol=1e-14)
    # <e_i, b_j> is symmetric in the two operands' roles only through the dot product:
    # swapping the columns of both e and b together leaves g unchanged
    gp, _ = oracle_mod.gauss_vjp(x, y, b[:, ::-1], e1[:, ::-1], 0.4)
    np.testing.assert_allclose(gp, g1, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("formula", ["gauss", "laplace"])
def test_kernel_lse_is_log_of_kernel_sum(oracle_mod, formula):
    # log sum_j k_ij exp(g_j) against the (pinned) kernel sum with b = exp(g)
    rng = np.random.default_rng(17)
    x = rng.uniform(0, 1, (10, 3)); y = rng.uniform(0, 1, (45, 3)); g = rng.normal(size=(45, 1))
    a, m = oracle_mod.kernel_lse(formula, x, y, g, 0.2)
    s, _ = oracle_mod.kernel_sum(formula, x, y, np.exp(g), sigma=0.2)
    np.testing.assert_allclose(a, np.log(s[:, 0]), rtol=1e-13)
    # and the row maximum is the log of the largest term k_ij exp(g_j)
    v, _, _ = oracle_mod.extreme(formula, "max", x, y, np.exp(g), param=0.2)
    np.testing.assert_allclose(m, np.log(v[:, 0]), rtol=1e-12, atol=1e-14)


def test_kernel_lse_gauss_is_sinkhorn_form(oracle_mod):
    # g_j - d / (2 sigma^2) is the Sinkhorn-form formula with eps = 2 sigma^2,
    # also far outside exp's range (g shifted by 1e4)
    rng = np.random.default_rng(18)
    x = rng.uniform(0, 1, (8, 2)); y = rng.uniform(0, 1, (30, 2)); g = rng.normal(size=(30, 1)) + 1e4
    a, m = oracle_mod.kernel_lse("gauss", x, y, g, 0.1)
    a2, m2 = oracle_mod.sinkhorn_lse(x, y, g, 2 * 0.1 ** 2)
    np.testing.assert_allclose(a, a2, rtol=1e-15)
    np.testing.assert_allclose(m, m2, rtol=1e-15)


def test_kernel_lse_laplace_two_points(oracle_mod):
    # closed form: log(exp(0 - 0) + exp(1 - 5/5)) = log 2 with |y_1 - x| = 5
    x = np.zeros((1, 2)); y = np.array([[0.0, 0.0], [3.0, 4.0]]); g = np.array([[0.0], [1.0]])
    a, m = oracle_mod.kernel_lse("laplace", x, y, g, 5.0)
    assert a[0] == pytest.approx(math.log(2.0), rel=1e-15)
    assert m[0] == 0.0


# ------------------------------------------------------------ min / max / arg-min

def test_extreme_hand_values(oracle_mod, hv):
    c = hv["extreme_small"]
    x, y, b = _a(c["x"]), _a(c["y"]), _a(c["b"])
    for key, formula, op, bb in (("sqdist_min", "sqdist", "min", None), ("sqdist_max", "sqdist", "max", None),
                                 ("gauss_max", "gauss", "max", b), ("gauss_min", "gauss", "min", b)):
        v, i, _ = oracle_mod.extreme(formula, op, x, y, bb, param=c["sigma"])
        assert v[0, 0] == pytest.approx(c["value"][key][0], rel=1e-14, abs=1e-15), key
        assert i[0, 0] == c["value"][key][1], key


def test_extreme_min_is_argkmin_k1(oracle_mod):
    # squared-distance min / arg-min against the brute-force-pinned arg-K-min
    # with K = 1, on integer coordinates full of exact ties
    rng = np.random.default_rng(12)
    x = rng.integers(-2, 3, (40, 3)).astype(np.float64); y = rng.integers(-2, 3, (60, 3)).astype(np.float64)
    v, i, _ = oracle_mod.extreme("sqdist", "min", x, y)
    idx, dist = oracle_mod.argkmin(x, y, 1)
    np.testing.assert_array_equal(i[:, 0], idx[:, 0])
    np.testing.assert_array_equal(v[:, 0], dist[:, 0])


def test_extreme_lse_formula_max_is_lse_row_max(oracle_mod):
    # the log-sum-exp routine's two-pass maximum m_i = max_j s_ij
    rng = np.random.default_rng(13)
    x = rng.uniform(0, 1, (9, 3)); y = rng.uniform(0, 1, (40, 3)); g = rng.normal(size=(40, 1))
    v, i, _ = oracle_mod.extreme("sinkhorn", "max", x, y, g, param=0.05)
    a, m = oracle_mod.sinkhorn_lse(x, y, g, 0.05)
    np.testing.assert_allclose(v[:, 0], m, rtol=1e-15)


@pytest.mark.parametrize("formula", ["gauss", "laplace", "sqdist"])
def test_extreme_sign_symmetry_and_ties(oracle_mod, formula):
    # min of F b = -(max of F (-b)), same (lowest) index; duplicated columns tie
    rng = np.random.default_rng(14)
    x = rng.uniform(0, 1, (11, 2)); y = rng.uniform(0, 1, (30, 2))
    y = np.concatenate([y, y[::-1]])   # every column appears twice
    b = rng.normal(size=(30, 3)); b = np.concatenate([b, b[::-1]])
    vmin, imin, s1 = oracle_mod.extreme(formula, "min", x, y, b, param=0.3)
    vmax, imax, s2 = oracle_mod.extreme(formula, "max", x, y, -b, param=0.3)
    np.testing.assert_array_equal(vmin, -vmax)
    np.testing.assert_array_equal(imin, imax)
    assert (imin < 30).all()   # the first copy of a tied column wins
    np.testing.assert_array_equal(s1, s2)


@pytest.mark.parametrize("op", ["min", "max"])
def test_extreme_components_are_independent(oracle_mod, op):
    # component e of an E-column call equals the one-column call on b[:, e]
    rng = np.random.default_rng(16)
    x = rng.uniform(0, 1, (10, 3)); y = rng.uniform(0, 1, (35, 3)); b = rng.normal(size=(35, 4))
    v, i, s = oracle_mod.extreme("gauss", op, x, y, b, param=0.25)
    for e in range(4):
        ve, ie, se = oracle_mod.extreme("gauss", op, x, y, b[:, [e]], param=0.25)
        np.testing.assert_array_equal(v[:, e], ve[:, 0])
        np.testing.assert_array_equal(i[:, e], ie[:, 0])


def test_extreme_gauss_max_is_nearest_point(oracle_mod):
    # with b = 1 the Gaussian is largest at the nearest point: exp(-d_min / 2 sigma^2)
    rng = np.random.default_rng(15)
    x = rng.uniform(0, 1, (12, 3)); y = rng.uniform(0, 1, (50, 3))
    v, i, _ = oracle_mod.extreme("gauss", "max", x, y, np.ones((50, 1)), param=0.2)
    idx, dist = oracle_mod.argkmin(x, y, 1)
    np.testing.assert_array_equal(i[:, 0], idx[:, 0])
    np.testing.assert_allclose(v[:, 0], np.exp(-dist[:, 0] / (2 * 0.2 ** 2)), rtol=1e-14)


def test_extreme_empty(oracle_mod):
    v, i, s = oracle_mod.extreme("sqdist", "min", np.zeros((2, 3)), np.zeros((0, 3)))
    assert np.isinf(v).all() and (v > 0).all() and (i == -1).all() and (s == 0).all()


# ---------------------------------------------------------------------- log-sum-exp

def test_lse_single_point(oracle_mod):
    x = _a([[0.1, 0.2, 0.3], [1.0, 0.0, -1.0]]); y = _a([[0.0, 0.0, 0.0]]); g = _a([[0.7]])
    a, _ = oracle_mod.sinkhorn_lse(x, y, g, 0.5)
    want = 0.7 - np.sum(x ** 2, 1) / 0.5
    np.testing.assert_allclose(a, want, rtol=1e-14)


def test_lse_eps_to_infinity_is_logsumexp_of_g(oracle_mod):
    rng = np.random.default_rng(9)
    x = rng.uniform(0, 1, (5, 3)); y = rng.uniform(0, 1, (50, 3)); g = rng.normal(size=(50, 1))
    a, _ = oracle_mod.sinkhorn_lse(x, y, g, 1e30)
    np.testing.assert_allclose(a, np.logaddexp.reduce(g[:, 0]), rtol=1e-14)


def test_lse_shift_and_large_offsets(oracle_mod):
    rng = np.random.default_rng(10)
    x = rng.uniform(0, 1, (7, 3)); y = rng.uniform(0, 1, (64, 3)); g = rng.normal(size=(64, 1))
    a, m = oracle_mod.sinkhorn_lse(x, y, g, 0.01)
    for c in (3.5, -1000.0, 1000.0):
        ac, mc = oracle_mod.sinkhorn_lse(x, y, g + c, 0.01)
        np.testing.assert_allclose(ac, a + c, rtol=1e-13, atol=1e-11)
        np.testing.assert_allclose(mc, m + c, rtol=1e-13, atol=1e-11)
    # log-sum-exp lies between the max and the max + log N
    assert np.all(a >= m - 1e-12) and np.all(a <= m + math.log(64) + 1e-12)


def test_lse_equals_log_of_gaussian_sum(oracle_mod):
    # With g_j = log b_j (b > 0) and eps = 2 sigma^2 the two formulas coincide:
    # log sum_j exp(log b_j - d/(2 sigma^2)) = log sum_j exp(-d/(2 sigma^2)) b_j.
    rng = np.random.default_rng(11)
    x = rng.uniform(0, 1, (9, 3)); y = rng.uniform(0, 1, (80, 3)); b = rng.uniform(0.1, 2.0, (80, 1))
    sigma = 0.2
    gs, _ = oracle_mod.kernel_sum("gauss", x, y, b, sigma=sigma)
    l, _ = oracle_mod.sinkhorn_lse(x, y, np.log(b), 2 * sigma ** 2)
    np.testing.assert_allclose(l, np.log(gs[:, 0]), rtol=1e-13)


# ------------------------------------------------------------------------- arg-K-min

def _brute_knn(x, y, K):
    d = ((x[:, None, :] - y[None, :, :]) ** 2).sum(-1)
    out = []
    for i in range(x.shape[0]):
        order = np.lexsort((np.arange(y.shape[0]), d[i]))  # primary: distance, then index
        out.append(order[:K])
    return np.array(out)


@pytest.mark.parametrize("K", [1, 3, 10, 57])
def test_argkmin_brute_force_with_ties(oracle_mod, K):
    rng = np.random.default_rng(12)
    # integer coordinates in a small box force many equal distances
    x = rng.integers(-2, 3, (23, 4)).astype(np.float64)
    y = rng.integers(-2, 3, (57, 4)).astype(np.float64)
    idx, dist = oracle_mod.argkmin(x, y, K)
    np.testing.assert_array_equal(idx, _brute_knn(x, y, K))
    # distances non-decreasing, and equal distances in increasing index order
    assert np.all(np.diff(dist, axis=1) >= 0)
    same = np.diff(dist, axis=1) == 0
    assert np.all(np.diff(idx, axis=1)[same] > 0)


def test_argkmin_full_sort_and_self_neighbour(oracle_mod):
    rng = np.random.default_rng(13)
    y = rng.normal(size=(40, 3))
    x = y[[5, 0, 39, 17]]
    idx, dist = oracle_mod.argkmin(x, y, 40)
    assert idx[:, 0].tolist() == [5, 0, 39, 17]
    assert np.all(dist[:, 0] == 0)
    np.testing.assert_array_equal(idx, _brute_knn(x, y, 40))
    for r in range(4):
        assert sorted(idx[r].tolist()) == list(range(40))


def test_argkmin_duplicate_points_lowest_index_first(oracle_mod):
    y = _a([[1, 1], [0, 0], [1, 1], [0, 0], [0, 0], [2, 2]])
    idx, _ = oracle_mod.argkmin(_a([[0, 0]]), y, 5)
    assert idx[0].tolist() == [1, 3, 4, 0, 2]


def test_argkmin_rejects_bad_k(oracle_mod):
    x = np.zeros((2, 2)); y = np.zeros((3, 2))
    with pytest.raises(ValueError):
        oracle_mod.argkmin(x, y, 4)
    with pytest.raises(ValueError):
        oracle_mod.argkmin(x, y, 0)


# ---------------------------------------------------------- block-sparse ranges

def _random_ranges(rng, M, N, n_rc, n_cc):
    """Row clusters covering part of [0, M) and, per cluster, sorted disjoint column ranges."""
    rcuts = np.sort(rng.choice(np.arange(1, M), n_rc * 2 - 1, replace=False))
    rcuts = np.concatenate([[0], rcuts, [M]])
    rows = [(int(rcuts[2 * i]), int(rcuts[2 * i + 1])) for i in range(n_rc)]   # gaps between clusters
    ccuts = np.concatenate([[0], np.sort(rng.choice(np.arange(1, N), n_cc - 1, replace=False)), [N]])
    cblocks = [(int(ccuts[k]), int(ccuts[k + 1])) for k in range(n_cc)]
    ptr, cr = [0], []
    for i in range(n_rc):
        keep = sorted(rng.choice(n_cc, rng.integers(0, n_cc + 1), replace=False))
        cr.extend(cblocks[k] for k in keep)
        ptr.append(len(cr))
    return np.array(rows), np.array(ptr), np.array(cr).reshape(-1, 2)


def _row_mask(rows, ptr, cr, M, N):
    mask = np.zeros((M, N), dtype=bool)
    covered = np.zeros(M, dtype=bool)
    for I, (r0, r1) in enumerate(rows):
        covered[r0:r1] = True
        for q in range(ptr[I], ptr[I + 1]):
            mask[r0:r1, cr[q][0]:cr[q][1]] = True
    return mask, covered


def test_ranges_full_cover_is_dense(oracle_mod):
    rng = np.random.default_rng(20)
    x = rng.uniform(0, 1, (30, 3)); y = rng.uniform(0, 1, (50, 3)); b = rng.normal(size=(50, 2))
    rows, ptr, cr = np.array([[0, 30]]), np.array([0, 1]), np.array([[0, 50]])
    a, n = oracle_mod.ranges_reduce("sum", x, y, b, rows, ptr, cr, formula="gauss", sigma=0.3)
    a2, n2 = oracle_mod.kernel_sum("gauss", x, y, b, sigma=0.3)
    np.testing.assert_array_equal(a, a2)
    idx, _ = oracle_mod.ranges_reduce("argkmin", x, y, None, rows, ptr, cr, K=4)
    idx2, _ = oracle_mod.argkmin(x, y, 4)
    np.testing.assert_array_equal(idx, idx2)


def test_ranges_sum_equals_masked_dense_rows(oracle_mod):
    # a_i over the allowed columns = the dense sum of row i with b zeroed
    # outside them; rows outside every cluster are 0
    rng = np.random.default_rng(21)
    M, N = 40, 60
    x = rng.uniform(0, 1, (M, 2)); y = rng.uniform(0, 1, (N, 2)); b = rng.normal(size=(N, 3))
    rows, ptr, cr = _random_ranges(rng, M, N, 4, 5)
    mask, covered = _row_mask(rows, ptr, cr, M, N)
    a, _ = oracle_mod.ranges_reduce("sum", x, y, b, rows, ptr, cr, formula="laplace", sigma=0.4)
    for i in range(M):
        ref, _ = oracle_mod.kernel_sum("laplace", x[i:i + 1], y, b * mask[i][:, None], sigma=0.4)
        np.testing.assert_allclose(a[i], ref[0], rtol=1e-13, atol=1e-15)
    assert (a[~covered] == 0).all()


def test_ranges_lse_equals_masked_log_weights(oracle_mod):
    # columns outside the pattern get log-weight -inf (their terms vanish)
    rng = np.random.default_rng(22)
    M, N = 35, 50
    x = rng.uniform(0, 1, (M, 3)); y = rng.uniform(0, 1, (N, 3)); g = rng.normal(size=(N, 1))
    rows, ptr, cr = _random_ranges(rng, M, N, 3, 4)
    mask, covered = _row_mask(rows, ptr, cr, M, N)
    a, _ = oracle_mod.ranges_reduce("lse", x, y, g, rows, ptr, cr, eps=0.05)
    for i in range(M):
        if not mask[i].any():
            assert a[i] == -np.inf
            continue
        gi = np.where(mask[i][:, None], g, -np.inf)
        keep = mask[i]
        ref, _ = oracle_mod.sinkhorn_lse(x[i:i + 1], y[keep], gi[keep], 0.05)
        assert a[i] == pytest.approx(ref[0], rel=1e-14)


def test_ranges_argkmin_maps_back_to_global_indices(oracle_mod):
    # indices are global column indices; a cluster with fewer than K columns pads with -1
    x = np.array([[0.0], [10.0]]); y = np.arange(12, dtype=np.float64).reshape(12, 1)
    rows, ptr, cr = np.array([[0, 1], [1, 2]]), np.array([0, 2, 3]), np.array([[8, 10], [2, 4], [11, 12]])
    idx, _ = oracle_mod.ranges_reduce("argkmin", x, y, None, rows, ptr, cr, K=3)
    np.testing.assert_array_equal(idx, [[2, 3, 8], [11, -1, -1]])


def _ranges_loss(oracle_mod, x, y, b, e, sigma, pat):
    # L = sum_i <e_i, a_i> with a the oracle's block-sparse Gaussian sum
    a, _ = oracle_mod.ranges_reduce("sum", x, y, b, *pat, formula="gauss", sigma=sigma)
    return float((a * e).sum())


def test_ranges_backward_matches_finite_differences(oracle_mod):
    # gradients of the masked sum in x, y (central differences) and b (exact:
    # L is linear in b), from the forward (row-cluster) pattern alone; rows
    # and columns the pattern never pairs get zero
    rng = np.random.default_rng(23)
    M, N, D, E, sigma = 14, 19, 2, 2, 0.3
    x = rng.uniform(0, 1, (M, D)); y = rng.uniform(0, 1, (N, D))
    b = rng.normal(size=(N, E)); e = rng.normal(size=(M, E))
    pat = _random_ranges(rng, M, N, 3, 4)
    gx, nx, gy, ny, gb, nb = oracle_mod.ranges_backward(x, y, b, e, sigma, *pat)
    mask, covered = _row_mask(*pat, M, N)
    h = 1e-5 * sigma
    for var, grad, scale in (("x", gx, nx.max()), ("y", gy, ny.max())):
        base = x if var == "x" else y
        for i in range(base.shape[0]):
            for k in range(D):
                p = base.copy(); p[i, k] += h
                m = base.copy(); m[i, k] -= h
                args_p = (p, y) if var == "x" else (x, p)
                args_m = (m, y) if var == "x" else (x, m)
                fd = (_ranges_loss(oracle_mod, *args_p, b, e, sigma, pat) -
                      _ranges_loss(oracle_mod, *args_m, b, e, sigma, pat)) / (2 * h)
                assert grad[i, k] == pytest.approx(fd, rel=1e-6, abs=1e-7 * scale)
    for j in range(N):
        for c in range(E):
            p = b.copy(); p[j, c] += 1.0
            fd = _ranges_loss(oracle_mod, x, y, p, e, sigma, pat) - _ranges_loss(oracle_mod, x, y, b, e, sigma, pat)
            assert gb[j, c] == pytest.approx(fd, rel=1e-10, abs=1e-12)
    assert (gx[~covered] == 0).all()
    assert (gy[~mask.any(0)] == 0).all() and (gb[~mask.any(0)] == 0).all()


def test_ranges_backward_full_cover_is_dense(oracle_mod):
    rng = np.random.default_rng(24)
    x = rng.uniform(0, 1, (25, 3)); y = rng.uniform(0, 1, (31, 3))
    b = rng.normal(size=(31, 3)); e = rng.normal(size=(25, 3))
    pat = (np.array([[0, 25]]), np.array([0, 2]), np.array([[0, 12], [12, 31]]))
    gx, _, gy, _, gb, _ = oracle_mod.ranges_backward(x, y, b, e, 0.4, *pat)
    np.testing.assert_allclose(gx, oracle_mod.gauss_vjp(x, y, b, e, 0.4)[0], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(gy, oracle_mod.gauss_vjp(y, x, e, b, 0.4)[0], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(gb, oracle_mod.kernel_sum("gauss", y, x, e, sigma=0.4)[0],
                               rtol=1e-12, atol=1e-14)
