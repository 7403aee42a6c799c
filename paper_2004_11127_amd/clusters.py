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
  so that no pair of points closer than the cutoff is dropped).

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
