"""Host-side construction of block-sparse patterns for kred_run_ranges.

The paper's library lets users specify cluster-wise block-sparsity patterns
(Sec. 3) together with a block-sparse truncation rule: points are grouped into
clusters, sorted so that each cluster is a contiguous range, and each cluster
of x interacts only with the clusters of y listed for it.  This module builds
such a pattern with numpy (setup work, outside the GPU hot path):

* grid_cluster: cluster labels from a grid of cubic cells;
* sort_by_labels: the permutation making each cluster contiguous, and its ranges;
* truncation_pattern: for each cluster of x, the ranges of the clusters of y
  whose cell centres lie within a cutoff distance (plus the cell diagonal,
  so that no pair of points closer than the cutoff is dropped);
* transpose_pattern: the same block set seen from the columns (column
  clusters, each with its row ranges), which the gradients in y and b of a
  block-sparse reduction sum over.

For a kernel that decays like the Gaussian exp(-|x - y|^2 / (2 sigma^2)), a
cutoff of c sigma drops only terms below exp(-c^2 / 2) of the largest.
"""
from __future__ import annotations

import numpy as np


def grid_cluster(points, cell, origin=None):
    """Cell index (int64) of each point on a grid of cubic cells of side `cell`."""
    p = np.asarray(points, dtype=np.float64)
    o = p.min(0) if origin is None else np.asarray(origin, dtype=np.float64)
    k = np.floor((p - o) / cell).astype(np.int64)
    k = np.maximum(k, 0)
    dims = k.max(0) + 1
    key = np.zeros(len(p), dtype=np.int64)
    for d in range(p.shape[1]):
        key = key * int(dims[d]) + k[:, d]
    return key, o, dims


def sort_by_labels(labels):
    """(order, unique labels, ranges): points[order] groups every label contiguously;
    ranges[i] = [start, end) of unique label i in the sorted order."""
    order = np.argsort(labels, kind="stable")
    uniq, start, count = np.unique(labels[order], return_index=True, return_counts=True)
    ranges = np.stack([start, start + count], 1).astype(np.int32)
    return order, uniq, ranges


def _cell_centres(keys, origin, dims, cell):
    D = len(dims)
    idx = np.empty((len(keys), D), dtype=np.int64)
    rest = keys.copy()
    for d in range(D - 1, -1, -1):
        idx[:, d] = rest % int(dims[d])
        rest //= int(dims[d])
    return origin + (idx + 0.5) * cell


def truncation_pattern(x, y, cell, cutoff):
    """Grid-cluster x and y, sort them, and keep the cluster pairs within cutoff.

    Returns a dict with the permutations `order_x`, `order_y` (apply them to x,
    y, b and undo on the output), the int32 arrays `row_ranges` (nr x 2),
    `col_ptr` (nr + 1) and `col_ranges` (nnz x 2) for kred_run_ranges on the
    sorted points, and `pairs`, the number of (i, j) pairs the pattern keeps.
    Adjacent kept clusters of y are merged into one column range.
    """
    x = np.asarray(x, dtype=np.float64); y = np.asarray(y, dtype=np.float64)
    origin = np.minimum(x.min(0), y.min(0))
    span = np.maximum(x.max(0), y.max(0)) - origin
    dims = np.floor(span / cell).astype(np.int64) + 1
    # one grid for both clouds (shared origin and extent)
    def keys(p):
        k = np.minimum(np.floor((p - origin) / cell).astype(np.int64), dims - 1)
        key = np.zeros(len(p), dtype=np.int64)
        for d in range(p.shape[1]):
            key = key * int(dims[d]) + k[:, d]
        return key
    kx, ky = keys(x), keys(y)
    ox, ux, rx = sort_by_labels(kx)
    oy, uy, ry = sort_by_labels(ky)
    cx = _cell_centres(ux, origin, dims, cell)
    cy = _cell_centres(uy, origin, dims, cell)
    reach = cutoff + cell * np.sqrt(x.shape[1])
    ptr = [0]
    col = []
    pairs = 0
    ny = ry[:, 1] - ry[:, 0]
    for i in range(len(ux)):
        keep = np.nonzero(((cy - cx[i]) ** 2).sum(1) <= reach * reach)[0]
        pairs += int(rx[i, 1] - rx[i, 0]) * int(ny[keep].sum())
        for k in keep:
            s, e = int(ry[k, 0]), int(ry[k, 1])
            if col and col[-1][1] == s and len(col) > ptr[-1]:
                col[-1][1] = e           # contiguous with the previous kept range
            else:
                col.append([s, e])
        ptr.append(len(col))
    return dict(order_x=ox, order_y=oy, row_ranges=rx.astype(np.int32),
                col_ptr=np.asarray(ptr, dtype=np.int32),
                col_ranges=np.asarray(col, dtype=np.int32).reshape(-1, 2), pairs=pairs)


def transpose_pattern(row_ranges, col_ptr, col_ranges, M, N):
    """The column-side view of a row-cluster pattern (kred_run_ranges's arrays).

    Returns int32 arrays (col_clusters (nc x 2), row_ptr (nc + 1), row_ranges_t
    (nnz x 2)) for kred_gauss_backward_ranges: column cluster J is the columns
    [col_clusters[J, 0], col_clusters[J, 1]) and its columns pair with the rows
    of row_ranges_t[row_ptr[J] : row_ptr[J + 1]], which are exactly the row
    clusters listing those columns.  Ranges are clamped to [0, M) x [0, N);
    row clusters must be disjoint.  Column clusters are the pieces between all
    range end points, merged where neighbours pair with the same rows; columns
    no row cluster lists belong to no column cluster.
    """
    rows = []   # (js, je, r0, r1) of every non-empty block
    for I in range(len(row_ranges)):
        r0 = min(max(int(row_ranges[I][0]), 0), M)
        r1 = min(max(int(row_ranges[I][1]), r0), M)
        if r1 <= r0:
            continue
        for q in range(int(col_ptr[I]), int(col_ptr[I + 1])):
            js = min(max(int(col_ranges[q][0]), 0), N)
            je = min(max(int(col_ranges[q][1]), js), N)
            if je > js:
                rows.append((js, je, r0, r1))
    cuts = np.unique(np.array([v for blk in rows for v in blk[:2]], dtype=np.int64))
    lists = [[] for _ in range(max(len(cuts) - 1, 0))]
    for js, je, r0, r1 in rows:
        for k in range(int(np.searchsorted(cuts, js)), int(np.searchsorted(cuts, je))):
            lists[k].append((r0, r1))
    clusters, ptr, rr = [], [0], []
    prev = None
    for k, lst in enumerate(lists):
        if not lst:
            prev = None
            continue
        merged = []
        for r0, r1 in sorted(lst):
            if merged and merged[-1][1] == r0:
                merged[-1][1] = r1
            else:
                merged.append([r0, r1])
        if prev is not None and prev == merged and clusters[-1][1] == int(cuts[k]):
            clusters[-1][1] = int(cuts[k + 1])   # same rows as the piece before: extend it
            continue
        clusters.append([int(cuts[k]), int(cuts[k + 1])])
        rr.extend(merged)
        ptr.append(len(rr))
        prev = merged
    return (np.asarray(clusters, dtype=np.int32).reshape(-1, 2),
            np.asarray(ptr, dtype=np.int32), np.asarray(rr, dtype=np.int32).reshape(-1, 2))
