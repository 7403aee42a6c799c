"""GPU parity of the exact bf16 arg-K-min kernel (16 < D <= 256) against the fp64 oracle.

On integer coordinates with |v| <= 256 and D max|v|^2 <= 2^22 the library
ranks columns on the bf16 matrix cores; every operand, product and partial
sum is then exact, so indices (lowest index on ties), K-min values and
nearest distances must equal the oracle's bit for bit.  The device-side guard
must send everything else (fractions, larger integers, larger sums) to the
fp32 kernel, and KRED_FLAG_DIRECT must keep the fp32 kernel.
"""
import numpy as np
import pytest

import oracle
from helpers import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx():
    import torch
    from paper_2004_11127_amd import kred
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    with kred.Context(0) as c:
        yield c


def _ints(rng, n, D, lo, hi):
    return rng.integers(lo, hi + 1, (n, D)).astype(np.float32)


def _run(ctx, reduction, x, y, K=1, C=0, flags=None):
    from paper_2004_11127_amd import kred
    fl = kred.FLAG_FAST if flags is None else flags
    ctx.profile_collect()
    out = host(ctx.run("sqdist", reduction, dev(x), dev(y), None, K=K, col_blocks=C,
                       flags=fl | kred.FLAG_PROFILE))
    return out, ctx.profile_collect()[2]


CASES = [
    # M, N, D, K, col_blocks, lo, hi
    (1, 1, 17, 1, 0, -8, 8),
    (65, 300, 32, 10, 0, -8, 8),
    (300, 2000, 64, 10, 0, -8, 8),
    (1000, 1500, 64, 10, 5, -8, 8),
    (129, 777, 128, 16, 0, -20, 20),
    (100, 900, 200, 4, 2, -3, 3),
    (70, 640, 64, 64, 1, -8, 8),
    (513, 1001, 40, 1, 3, -100, 100),
    (64, 64, 64, 64, 0, 0, 1),
    (200, 3000, 256, 10, 0, -2, 2),
    (257, 999, 33, 16, 7, -256, 256),   # |v| = 256 allowed while 33 * 256^2 <= 2^22
    (300, 1200, 64, 12, 0, -8, 8),
    (200, 900, 96, 7, 3, -8, 8),
    (4000, 3000, 64, 9, 0, -4, 4),      # many row blocks, dense ties
]


@pytest.mark.parametrize("M,N,D,K,C,lo,hi", CASES)
def test_exact_argkmin_bit_exact(ctx, M, N, D, K, C, lo, hi):
    rng = np.random.default_rng(M + 7 * N + D + K)
    x = _ints(rng, M, D, lo, hi); y = _ints(rng, N, D, lo, hi)
    y[N // 2:N // 2 + N // 8] = y[:N // 8]   # exact ties between columns
    out, name = _run(ctx, "argkmin", x, y, K=K, C=C)
    assert name == "knn_bf16_kernel"
    ref, _ = oracle.argkmin(x, y, K)
    np.testing.assert_array_equal(out, ref)


@pytest.mark.parametrize("M,N,D,K,C", [(300, 2000, 64, 10, 0), (129, 777, 128, 16, 3), (65, 70, 20, 64, 0)])
def test_exact_kmin_values_bit_exact(ctx, M, N, D, K, C):
    rng = np.random.default_rng(M + N + D)
    x = _ints(rng, M, D, -8, 8); y = _ints(rng, N, D, -8, 8)
    out, name = _run(ctx, "kmin", x, y, K=K, C=C)
    assert name == "knn_bf16_kernel"
    _, ref = oracle.argkmin(x, y, K)
    np.testing.assert_array_equal(out, ref.astype(np.float32))


@pytest.mark.parametrize("red", ["min", "argmin"])
def test_exact_nearest_bit_exact(ctx, red):
    rng = np.random.default_rng(5)
    x = _ints(rng, 700, 48, -8, 8); y = _ints(rng, 2500, 48, -8, 8)
    out, name = _run(ctx, red, x, y)
    assert name == "knn_bf16_kernel"
    val, idx, _ = oracle.extreme("sqdist", "min", x, y)
    if red == "min":
        np.testing.assert_array_equal(out, val.astype(np.float32))
    else:
        np.testing.assert_array_equal(out, idx.astype(np.int32))


FALLBACK = [
    # what makes the guard refuse, and the data
    ("fraction", lambda r: _ints(r, 300, 64, -8, 8) + np.float32(0.5) * (r.random((300, 64)) < 0.01)),
    ("large integer", lambda r: _ints(r, 300, 24, -300, 300)),
    # 80 * 256^2 > 2^22, while 3 * 80 * 256^2 < 2^24 keeps the fp32 kernel exact
    ("large sum", lambda r: _ints(r, 300, 80, -256, 256)),
]


@pytest.mark.parametrize("why,make", FALLBACK, ids=[f[0] for f in FALLBACK])
def test_guard_falls_back_to_fp32(ctx, why, make):
    rng = np.random.default_rng(11)
    x = make(rng).astype(np.float32)
    y = make(rng).astype(np.float32)[:250]
    out, name = _run(ctx, "argkmin", x, y, K=5)
    assert name == "mfma_kernel"
    ref, ref_d = oracle.argkmin(x, y, 5)
    if why == "fraction":
        # not exact in fp32 either: each index must be a valid k-th nearest
        got = ((x[:, None, :].astype(np.float64) - y[out].astype(np.float64)) ** 2).sum(-1)
        np.testing.assert_allclose(got, ref_d, rtol=1e-5, atol=1e-3)
    else:
        np.testing.assert_array_equal(out, ref)


@pytest.mark.parametrize("K", [7, 10, 12])
def test_direct_flag_keeps_fp32_kernel(ctx, K):
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(3 + K)
    x = _ints(rng, 200, 64, -8, 8); y = _ints(rng, 1000, 64, -8, 8)
    out, name = _run(ctx, "argkmin", x, y, K=K, flags=kred.FLAG_DIRECT)
    assert name == "mfma_kernel"
    np.testing.assert_array_equal(out, oracle.argkmin(x, y, K)[0])


def test_exact_path_matches_fp32_path_and_repeats(ctx):
    # same data through both kernels, twice through the exact one (the guard is reset per call)
    from paper_2004_11127_amd import kred
    rng = np.random.default_rng(9)
    x = _ints(rng, 777, 64, -8, 8); y = _ints(rng, 4000, 64, -8, 8)
    a, na = _run(ctx, "argkmin", x, y, K=10)
    b, nb = _run(ctx, "argkmin", x, y, K=10, flags=kred.FLAG_DIRECT)
    xf = x + np.float32(0.25)   # fractions: the next call must fall back
    c, nc = _run(ctx, "argkmin", xf, y, K=10)
    d, nd = _run(ctx, "argkmin", x, y, K=10)
    assert (na, nb, nc, nd) == ("knn_bf16_kernel", "mfma_kernel", "mfma_kernel", "knn_bf16_kernel")
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(a, d)
