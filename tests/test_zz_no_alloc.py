"""kred_run_noalloc: the same results as kred_run from the library's fixed scratch.

Each case runs twice in a row through the no-allocation entry point, the
second time on a smaller input, and compares with kred_run on the same inputs
(the same kernels and plan, so the same bits) and, for one case per family,
with the fp64 oracle.  Calls needing more than the fixed scratch, and profiled
calls, are refused before anything runs.
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


def _data(seed, M, N, D, E, integer=False):
    rng = np.random.default_rng(seed)
    if integer:
        x = rng.integers(-8, 9, (M, D)).astype(np.float32)
        y = rng.integers(-8, 9, (N, D)).astype(np.float32)
    else:
        x = rng.uniform(0, 1, (M, D)).astype(np.float32)
        y = rng.uniform(0, 1, (N, D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32) if E else None
    return x, y, b


CASES = [
    # formula, reduction, D, E, params, (M, N) of the first and second call
    ("gauss", "sum", 3, 1, dict(sigma=0.05, flags=4), (3000, 5000), (1000, 2000)),      # matrix-core exponent
    ("gauss", "sum", 3, 1, dict(sigma=0.1), (2000, 3000), (700, 900)),                  # direct form
    ("gauss", "sum", 5, 17, dict(sigma=0.3, col_blocks=7), (1500, 2500), (300, 400)),   # two E-slices, split
    ("gauss_gradx", "sum", 3, 1, dict(sigma=0.05), (2000, 3000), (500, 800)),
    ("sinkhorn", "lse", 3, 1, dict(eps=0.01, flags=4), (2000, 3000), (600, 700)),
    ("sqdist", "argkmin", 16, 0, dict(K=10), (1500, 4000), (400, 1000)),
    ("sqdist", "argkmin", 3, 0, dict(K=8, flags=4), (1500, 4000), (400, 1000)),        # K-lists on the matrix cores
    ("gauss", "sum", 64, 16, dict(sigma=1.0), (1500, 2500), (500, 600)),               # large D, fp32 matrix cores
    ("gauss", "sum", 64, 16, dict(sigma=1.0, flags=4), (1500, 2500), (500, 600)),      # large D, split bf16 kernel
    ("gauss_gradx", "sum", 40, 1, dict(sigma=1.0), (1200, 2000), (300, 500)),          # large D, signal chunks
    ("sinkhorn", "lse", 48, 1, dict(eps=1.0), (1200, 2000), (300, 500)),
    ("sinkhorn", "lse", 48, 1, dict(eps=1.0, flags=4), (1200, 2000), (300, 500)),      # large D, split log-sum-exp
    ("gauss", "sum", 128, 40, dict(sigma=1.0, flags=4), (900, 1300), (300, 400)),      # split, 64 signal columns
    ("gauss_gradx", "sum", 64, 1, dict(sigma=1.0, flags=4), (1500, 2500), (400, 600)),  # 65th column in the first launch
    ("gauss", "max", 24, 3, dict(sigma=1.0), (800, 1500), (200, 300)),
]


@pytest.mark.parametrize("formula,reduction,D,E,kw,first,second", CASES)
def test_noalloc_matches_run(ctx, formula, reduction, D, E, kw, first, second):
    for call, (M, N) in enumerate((first, second)):
        x, y, b = _data(M + N + D + call, M, N, D, E)
        xd, yd = dev(x), dev(y)
        bd = dev(b) if b is not None else None
        ref = host(ctx.run(formula, reduction, xd, yd, bd, **kw))
        got = host(ctx.run_noalloc(formula, reduction, xd, yd, bd, **kw))
        assert got.shape == ref.shape
        np.testing.assert_array_equal(got, ref)
        if call == 1 and reduction == "sum" and formula == "gauss" and D <= 16:
            oref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=kw["sigma"])
            assert norm_err(got, oref, norm) <= SUM_TOL


def test_noalloc_exact_knn_guard(ctx):
    # the exact bf16 k-NN kernel's device guard also lives in the fixed scratch
    from paper_2004_11127_amd import kred
    for M, N in ((1000, 3000), (300, 700)):
        x, y, _ = _data(M + N, M, N, 64, 0, integer=True)
        got = host(ctx.run_noalloc("sqdist", "argkmin", dev(x), dev(y), None, K=10,
                                   flags=kred.FLAG_FAST))
        idx, _ = oracle.argkmin(x, y, 10)
        np.testing.assert_array_equal(got, idx.astype(np.int32))


def test_noalloc_interleaved_with_run(ctx):
    # the allocating entry point and the fixed scratch do not disturb each other
    x, y, b = _data(5, 2500, 4000, 3, 1)
    xd, yd, bd = dev(x), dev(y), dev(b)
    a1 = host(ctx.run_noalloc("gauss", "sum", xd, yd, bd, sigma=0.07))
    a2 = host(ctx.run("gauss", "sum", xd, yd, bd, sigma=0.07, col_blocks=5))
    a3 = host(ctx.run_noalloc("gauss", "sum", xd, yd, bd, sigma=0.07))
    np.testing.assert_array_equal(a1, a3)
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.07)
    assert norm_err(a1, ref, norm) <= SUM_TOL and norm_err(a2, ref, norm) <= SUM_TOL


def test_noalloc_refuses_too_large_and_profiled(ctx):
    import torch
    from paper_2004_11127_amd import kred
    M, N, D = 100, 1_000_000, 16   # the packed y alone is 68 MB, more than the fixed 32 MiB
    x = torch.zeros((M, D), device="cuda"); y = torch.zeros((N, D), device="cuda")
    b = torch.zeros((N, 1), device="cuda")
    out = torch.full((M, 1), 7.0, device="cuda")
    assert kred.load().kred_scratch_bytes(0, 0, kred.make_params(sigma=1.0), M, N, D, 1) > \
        kred.NOALLOC_SCRATCH_BYTES
    with pytest.raises(kred.KredError) as e:
        ctx.run_noalloc("gauss", "sum", x, y, b, out=out, sigma=1.0)
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert (out == 7.0).all()   # nothing ran
    small = torch.zeros((10, D), device="cuda")
    with pytest.raises(kred.KredError) as e:
        ctx.run_noalloc("gauss", "sum", small, small, torch.zeros((10, 1), device="cuda"),
                        sigma=1.0, flags=kred.FLAG_PROFILE)
    assert e.value.status == 1
