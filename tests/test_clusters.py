"""Host-side block-sparse pattern construction (CPU only)."""
import numpy as np

from paper_2004_11127_amd import clusters


def test_sort_by_labels_groups_contiguously():
    lab = np.array([3, 1, 3, 0, 1, 3])
    order, uniq, ranges = clusters.sort_by_labels(lab)
    np.testing.assert_array_equal(uniq, [0, 1, 3])
    np.testing.assert_array_equal(ranges, [[0, 1], [1, 3], [3, 6]])
    for u, (s, e) in zip(uniq, ranges):
        assert (lab[order[s:e]] == u).all()


def test_truncation_pattern_keeps_every_close_pair():
    rng = np.random.default_rng(0)
    x = rng.uniform(0, 1, (400, 3)); y = rng.uniform(0, 1, (500, 3))
    pat = clusters.truncation_pattern(x, y, cell=0.2, cutoff=0.25)
    xs, ys = x[pat["order_x"]], y[pat["order_y"]]
    kept = np.zeros((400, 500), dtype=bool)
    for I, (r0, r1) in enumerate(pat["row_ranges"]):
        for q in range(pat["col_ptr"][I], pat["col_ptr"][I + 1]):
            c0, c1 = pat["col_ranges"][q]
            kept[r0:r1, c0:c1] = True
    d = np.sqrt(((xs[:, None, :] - ys[None, :, :]) ** 2).sum(-1))
    assert kept[d <= 0.25].all()                 # nothing within the cutoff is dropped
    assert kept.sum() == pat["pairs"]
    assert kept.sum() < kept.size                # and something is dropped
    # ranges of a cluster are sorted and disjoint
    for I in range(len(pat["row_ranges"])):
        cr = pat["col_ranges"][pat["col_ptr"][I]:pat["col_ptr"][I + 1]]
        assert (cr[:, 0] < cr[:, 1]).all() and (cr[1:, 0] >= cr[:-1, 1]).all()


def _pattern_mask(rows, ptr, cr, M, N):
    """(M, N) mask of a row-cluster pattern, ranges clamped as the library does."""
    mask = np.zeros((M, N), dtype=bool)
    for I, (a, b) in enumerate(rows):
        r0 = min(max(int(a), 0), M); r1 = min(max(int(b), r0), M)
        for q in range(ptr[I], ptr[I + 1]):
            c0 = min(max(int(cr[q][0]), 0), N); c1 = min(max(int(cr[q][1]), c0), N)
            mask[r0:r1, c0:c1] = True
    return mask


def _random_pattern(rng, M, N, n_rc, n_cc):
    rc = np.sort(rng.choice(np.arange(1, M), 2 * n_rc - 1, replace=False))
    rc = np.concatenate([[0], rc, [M]])
    rows = np.array([[rc[2 * i], rc[2 * i + 1]] for i in range(n_rc)])
    cc = np.concatenate([[0], np.sort(rng.choice(np.arange(1, N), n_cc - 1, replace=False)), [N]])
    ptr, cr = [0], []
    for i in range(n_rc):
        keep = np.nonzero(rng.uniform(size=n_cc) < 0.4)[0]
        cr.extend([cc[k], cc[k + 1]] for k in keep)
        ptr.append(len(cr))
    return rows, np.array(ptr), np.array(cr).reshape(-1, 2)


def test_transpose_pattern_keeps_the_same_blocks():
    rng = np.random.default_rng(3)
    for M, N, n_rc, n_cc in [(50, 70, 5, 8), (200, 90, 30, 12), (17, 300, 3, 40)]:
        rows, ptr, cr = _random_pattern(rng, M, N, n_rc, n_cc)
        # ranges reaching outside [0, N), and an empty cluster, are clamped and skipped
        cr = np.concatenate([cr, [[N - 3, N + 50], [-9, 2]]])
        ptr = np.concatenate([ptr, [len(cr)]])
        rows = np.concatenate([rows, [[M - 1, M + 4]]])
        rows[0] = [rows[0][0], rows[0][0]]
        cc, rp, rt = clusters.transpose_pattern(rows, ptr, cr, M, N)
        assert cc.dtype == np.int32 and rp.dtype == np.int32 and rt.dtype == np.int32
        assert rp.shape == (len(cc) + 1,) and rp[-1] == len(rt)
        np.testing.assert_array_equal(_pattern_mask(cc, rp, rt, N, M).T,
                                      _pattern_mask(rows, ptr, cr, M, N))
        # column clusters are disjoint and sorted; each lists sorted, disjoint row ranges
        assert (cc[:, 0] < cc[:, 1]).all() and (cc[1:, 0] >= cc[:-1, 1]).all()
        for J in range(len(cc)):
            r = rt[rp[J]:rp[J + 1]]
            assert len(r) > 0 and (r[:, 0] < r[:, 1]).all() and (r[1:, 0] > r[:-1, 1]).all()


def test_transpose_pattern_of_a_truncation_rule():
    rng = np.random.default_rng(4)
    x = rng.uniform(0, 1, (300, 2)); y = rng.uniform(0, 1, (260, 2))
    pat = clusters.truncation_pattern(x, y, cell=0.15, cutoff=0.2)
    cc, rp, rt = clusters.transpose_pattern(pat["row_ranges"], pat["col_ptr"], pat["col_ranges"],
                                            300, 260)
    fwd = _pattern_mask(pat["row_ranges"], pat["col_ptr"], pat["col_ranges"], 300, 260)
    np.testing.assert_array_equal(_pattern_mask(cc, rp, rt, 260, 300).T, fwd)
    assert fwd.sum() == pat["pairs"]


def test_transpose_pattern_empty():
    cc, rp, rt = clusters.transpose_pattern(np.zeros((0, 2)), np.zeros(1), np.zeros((0, 2)), 10, 10)
    assert cc.shape == (0, 2) and rp.tolist() == [0] and rt.shape == (0, 2)
