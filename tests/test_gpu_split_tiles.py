"""GPU parity of the 32x32-tile split kernel (17 <= D <= 128) at every tile count: sums and log-sum-exp.

The kernel walks each column block in 32-column tiles through four sets of
LDS buffers (the loop unrolled by four, two tiles in flight, the pending
tile finished one step later with 16 signal columns and in place with 32
or 64), so a column block of 1 to 9 tiles meets every entry and exit of that
loop; N not a multiple of 16 or 32 leaves a partial last tile.  Workgroups
hold 256 rows (128 at D <= 32 and for the log-sum-exp at D <= 64), so M = 300
leaves a ragged last one.  Same bar as the other
sum and log-sum-exp tests: error normalised by sum_j |k_ij b_j| (sums), or
absolute in the log domain (log-sum-exp), at most 1e-4 against the fp64
oracle, and the kernel that ran is asserted.
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


def _data(M, N, D, E, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((M, D)) / np.sqrt(D)).astype(np.float32)
    y = (rng.standard_normal((N, D)) / np.sqrt(D)).astype(np.float32)
    b = rng.standard_normal((N, E)).astype(np.float32)
    return x, y, b


# (D, E): 16 signal columns (pipelined), 32 and 64 (finished in place), E
# below a block; D = 128, 64 and 32 (the three padded widths), and odd D
WIDTHS = [(128, 16), (128, 40), (100, 64), (64, 16), (64, 20), (40, 3), (32, 16), (32, 64), (24, 1)]
# columns: 1 to 9 tiles, full and partial last tiles
COLS = [1, 17, 32, 33, 64, 95, 128, 129, 160, 200, 257, 288]


@pytest.mark.parametrize("N", COLS)
@pytest.mark.parametrize("D,E", WIDTHS)
def test_split_kernel_tile_counts(ctx, D, E, N):
    from paper_2004_11127_amd import kred
    M = 300
    x, y, b = _data(M, N, D, E, seed=D * 1000 + E * 10 + N)
    ctx.profile_collect()
    out = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=1.0, col_blocks=1,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == "mfma_split_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=1.0)
    assert out.shape == (M, E)
    assert norm_err(out, ref, norm) <= SUM_TOL


@pytest.mark.parametrize("C", [2, 3, 8])
@pytest.mark.parametrize("D,E", [(128, 16), (128, 64), (64, 16), (32, 16)])
def test_split_kernel_column_blocks(ctx, D, E, C):
    # several column blocks (partials combined in a second pass), each with a
    # few tiles; C = 8 is the one-block-per-XCD choice
    from paper_2004_11127_amd import kred
    M, N = 520, 1000
    x, y, b = _data(M, N, D, E, seed=7 * C + D + E)
    ctx.profile_collect()
    out = host(ctx.run("gauss", "sum", dev(x), dev(y), dev(b), sigma=0.9, col_blocks=C,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == "mfma_split_kernel"
    ref, norm = oracle.kernel_sum("gauss", x, y, b, sigma=0.9)
    assert norm_err(out, ref, norm) <= SUM_TOL


def test_split_kernel_segments_restart(ctx):
    # block-sparse: many short column ranges per row cluster, so each
    # workgroup walks several segments (its buffers restart at each one), with
    # 16, 32 and 64 signal columns
    from paper_2004_11127_amd import kred
    M, N, D = 600, 1500, 128
    rng = np.random.default_rng(11)
    rr = np.array([[0, 260], [260, 300], [310, 600]], dtype=np.int32)
    cuts = np.sort(rng.choice(np.arange(1, N), size=24, replace=False))
    edges = np.concatenate([[0], cuts, [N]])
    spans = [(int(edges[k]), int(edges[k + 1])) for k in range(len(edges) - 1)]
    keep = [[s for k, s in enumerate(spans) if (k + i) % 3 != 0] for i in range(len(rr))]
    cp = np.cumsum([0] + [len(k) for k in keep]).astype(np.int32)
    cr = np.array([s for k in keep for s in k], dtype=np.int32)
    for E in (16, 32, 64):
        x, y, b = _data(M, N, D, E, seed=E)
        ctx.profile_collect()
        out = host(ctx.run_ranges("gauss", "sum", dev(x), dev(y), dev(b), dev(rr), dev(cp), dev(cr),
                                  sigma=1.0, col_blocks=2, flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
        assert ctx.profile_collect()[2] == "mfma_split_kernel"
        ref, norm = oracle.ranges_reduce("sum", x, y, b, rr, cp, cr, formula="gauss", sigma=1.0)
        assert norm_err(out, ref, norm) <= SUM_TOL
        assert (out[300:310] == 0).all()   # rows in no cluster


# ------------------------------------------------------------- log-sum-exp
# The Gaussian and Sinkhorn log-sum-exp take the same kernel at D = 17..128
# (bar: 1e-4 absolute in the log domain, as every LSE test)
def _lse_data(M, N, D, seed):
    # uniform in a box of side sqrt(32 / D) (the squared spread of the unit
    # cube at D = 32), so that the guard's L stays well inside the split
    # limit at every D here (about 15 against 24 at D = 128)
    spread = float(np.sqrt(32.0 / D))
    rng = np.random.default_rng(seed)
    x = (spread * rng.uniform(size=(M, D))).astype(np.float32)
    y = (spread * rng.uniform(size=(N, D))).astype(np.float32)
    y[:, 0] += 0.3
    g = rng.standard_normal((N, 1)).astype(np.float32)
    return x, y, g


@pytest.mark.parametrize("N", [1, 17, 32, 33, 95, 160, 257, 288])
@pytest.mark.parametrize("formula,D", [("sinkhorn", 64), ("sinkhorn", 128), ("gauss", 100), ("sinkhorn", 40),
                                           ("sinkhorn", 32), ("gauss", 20)])
def test_split_lse_tile_counts(ctx, formula, D, N):
    from paper_2004_11127_amd import kred
    from helpers import LSE_TOL, lse_err
    M = 300
    x, y, g = _lse_data(M, N, D, seed=D + N)
    kw = dict(eps=1.0) if formula == "sinkhorn" else dict(sigma=0.7)
    ctx.profile_collect()
    out = host(ctx.run(formula, "lse", dev(x), dev(y), dev(g), col_blocks=1,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE, **kw))
    assert ctx.profile_collect()[2] == "mfma_split_kernel"
    ref, m = (oracle.sinkhorn_lse(x, y, g, 1.0) if formula == "sinkhorn"
              else oracle.kernel_lse("gauss", x, y, g, 0.7))
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


@pytest.mark.parametrize("C", [0, 2, 8])
@pytest.mark.parametrize("D", [32, 64, 128])
def test_split_lse_column_blocks(ctx, D, C):
    from paper_2004_11127_amd import kred
    from helpers import LSE_TOL, lse_err
    M, N = 530, 1100
    x, y, g = _lse_data(M, N, D, seed=3 * C + D)
    ctx.profile_collect()
    out = host(ctx.run("sinkhorn", "lse", dev(x), dev(y), dev(g), eps=0.8, col_blocks=C,
                       flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
    assert ctx.profile_collect()[2] == "mfma_split_kernel"
    ref, m = oracle.sinkhorn_lse(x, y, g, 0.8)
    assert lse_err(out[:, 0], ref, m) <= LSE_TOL


def test_split_lse_segments_and_empty_rows(ctx):
    # block-sparse: many short segments per cluster; rows in no cluster are -inf
    from paper_2004_11127_amd import kred
    from helpers import LSE_TOL, lse_err
    M, N, D = 600, 1500, 64
    x, y, g = _lse_data(M, N, D, seed=5)
    rr = np.array([[0, 260], [260, 300], [310, 600]], dtype=np.int32)
    rng = np.random.default_rng(12)
    cuts = np.sort(rng.choice(np.arange(1, N), size=24, replace=False))
    edges = np.concatenate([[0], cuts, [N]])
    spans = [(int(edges[k]), int(edges[k + 1])) for k in range(len(edges) - 1)]
    keep = [[s for k, s in enumerate(spans) if (k + i) % 3 != 0] for i in range(len(rr))]
    cp = np.cumsum([0] + [len(k) for k in keep]).astype(np.int32)
    cr = np.array([s for k in keep for s in k], dtype=np.int32)
    for C in (1, 3):
        ctx.profile_collect()
        out = host(ctx.run_ranges("sinkhorn", "lse", dev(x), dev(y), dev(g), dev(rr), dev(cp), dev(cr),
                                  eps=0.5, col_blocks=C, flags=kred.FLAG_FAST | kred.FLAG_PROFILE))
        assert ctx.profile_collect()[2] == "mfma_split_kernel"
        ref, m = oracle.ranges_reduce("lse", x, y, g, rr, cp, cr, eps=0.5)
        live = np.isfinite(ref)
        assert lse_err(out[live, 0], ref[live], m[live]) <= LSE_TOL, C
        assert np.isneginf(out[300:310, 0]).all()
