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
