"""GPU parity of the one-launch Gaussian sum (D <= 4, E <= 4, below 2^28 pairs).

The kernel reads y and b straight into LDS, forms the pair term on the matrix
cores within each workgroup's own accuracy bound (or in the direct form beyond
it), and lets the last workgroup of each row block add the column blocks'
partials, resetting its counter for the next call.  Cases: every D and E,
ragged sizes, one and many column blocks, repeated calls with different
shapes (the counters must be back at zero), wide data that sends every
workgroup to the direct form, data where only some workgroups take it, the
c1 workload at full size, and the no-allocation entry point.  Bar: 1e-4 of
sum_j |k_ij b_je| per element.
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


def _run(ctx, x, y, b, sigma, **kw):
    from paper_2004_11127_amd import kred
    ctx.profile_collect()
    out = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=sigma,
                       flags=kw.pop("flags", 0) | kred.FLAG_PROFILE, **kw))
    return out, ctx.profile_collect()[2]


CASES = [
    # M, N, D, E, sigma, col_blocks
    (1037, 3005, 3, 1, 0.1, 0),
    (1037, 3005, 3, 1, 0.1, 1),      # raised to the 1024-column minimum (3 blocks)
    (300, 900, 3, 1, 0.1, 1),        # one column block: no partials, no counters
    (129, 17, 1, 1, 0.3, 0),
    (2000, 5000, 2, 2, 0.05, 0),
    (1500, 4000, 4, 3, 0.2, 7),
    (777, 2222, 4, 4, 0.15, 0),
    (1, 5000, 3, 2, 0.1, 0),         # a single row
    (4096, 1, 2, 1, 0.1, 0),         # a single column
]


@pytest.mark.parametrize("M,N,D,E,sigma,C", CASES)
def test_small_sum_parity(ctx, M, N, D, E, sigma, C):
    rng = np.random.default_rng(M + 7 * N + D + E)
    x = rng.uniform(0, 1, (M, D)).astype(np.float32)
    y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    out, name = _run(ctx, x, y, b, sigma, col_blocks=C)
    assert name == "small_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=sigma)
    assert out.shape == (M, E)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_repeated_calls_reset_the_counters(ctx):
    # alternating shapes and column-block counts: a counter left above zero by
    # one call would make the next call's last workgroup combine too early
    rng = np.random.default_rng(5)
    shapes = [(3000, 6000, 12), (500, 2500, 0), (3000, 6000, 3), (128, 9000, 0)] * 2
    for M, N, C in shapes:
        x = rng.uniform(0, 1, (M, 3)).astype(np.float32)
        y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
        b = rng.standard_normal((N, 1)).astype(np.float32)
        out, name = _run(ctx, x, y, b, 0.1, col_blocks=C)
        assert name == "small_kernel"
        ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.1)
        assert norm_err(out, ref, norm) <= SUM_TOL, (M, N, C)


def test_wide_data_takes_the_direct_form(ctx):
    # spread 1e3 against sigma 0.05: L far above every limit, so every
    # workgroup forms the pair term directly; half of x are points of y, whose
    # self-pairs carry the sums
    rng = np.random.default_rng(11)
    N, M = 4000, 1200
    y = (1000 * rng.uniform(0, 1, (N, 3))).astype(np.float32)
    x = np.concatenate([y[:M // 2], 1000 * rng.uniform(0, 1, (M - M // 2, 3))]).astype(np.float32)
    b = rng.standard_normal((N, 2)).astype(np.float32)
    out, name = _run(ctx, x, y, b, 0.05)
    assert name == "small_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.05)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_mixed_workgroups(ctx):
    # rows sorted so that some row blocks sit inside the unit cube (matrix
    # cores) and some far outside it (direct form); columns in the unit cube
    # plus a far cluster
    rng = np.random.default_rng(13)
    N, M = 3000, 2048
    y = np.concatenate([rng.uniform(0, 1, (N - 300, 3)), 50 + rng.uniform(0, 1, (300, 3))])
    x = np.concatenate([rng.uniform(0, 1, (1024, 3)), 50 + rng.uniform(0, 1, (1024, 3))])
    x, y = x.astype(np.float32), y.astype(np.float32)
    b = rng.standard_normal((N, 1)).astype(np.float32)
    out, name = _run(ctx, x, y, b, 0.1)
    assert name == "small_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.1)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_c1_full_size(ctx):
    from paper_2004_11127_amd import inputs
    w = inputs.uniform_gauss(M=10_000, N=10_000, D=3, E=1, sigma=0.1, seed=0)
    out, name = _run(ctx, w.x, w.y, w.b, w.sigma)
    assert name == "small_kernel"
    ref, norm = oracle.kernel_sum("gauss", w.x, w.y, w.b, sigma=w.sigma)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_flags_keep_the_other_paths(ctx):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(3)
    x = rng.uniform(0, 1, (1000, 3)).astype(np.float32)
    y = rng.uniform(0, 1, (2000, 3)).astype(np.float32)
    b = rng.standard_normal((2000, 1)).astype(np.float32)
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.1)
    out, name = _run(ctx, x, y, b, 0.1, flags=kred.FLAG_DIRECT)
    assert name == "sum_kernel"
    assert norm_err(out, ref, norm) <= SUM_TOL
    out, name = _run(ctx, x, y, b, 0.1, flags=kred.FLAG_FAST)
    assert name == "fast_kernel"
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_noalloc_matches(ctx):
    # the no-allocation entry point keeps the counters in its fixed scratch
    rng = np.random.default_rng(17)
    for M, N in [(2500, 7000), (300, 500), (2500, 7000)]:
        x = rng.uniform(0, 1, (M, 3)).astype(np.float32)
        y = rng.uniform(0, 1, (N, 3)).astype(np.float32)
        b = rng.standard_normal((N, 2)).astype(np.float32)
        a = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=0.1))
        n = host(ctx.run_noalloc("gauss", "sum", dev(x), dev(y), dev(b), sigma=0.1))
        np.testing.assert_array_equal(a, n)
