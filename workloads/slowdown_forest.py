"""Seeded tree ensembles standing in for the paper's trained slowdown predictor.

The paper predicts the slowdown of a compute kernel overlapped by a
collective with an XGBoost regressor (Sec. 6) over communication details and
kernel metrics (Table 4), trees at most 12 deep (Table 5).  Neither the model
nor its profiling dataset is available, so these ensembles are synthetic:
random splits over the same kind of features, small leaf values around a
base score.  They are inputs only; nothing here predicts anything.

An ensemble is a dict:
    nodes          TREE_NODE_DTYPE [n_nodes]  feature (-1 leaf), left, right,
                                              value (Q16 leaf contribution),
                                              threshold (left when x[feature] < threshold)
    roots          int32 [n_trees]
    base           int   base score (Q16)
    class_metrics  int64 [8, 4]  per kernel class: compute throughput, memory
                                 throughput, achieved occupancy, L2 hit rate (per mille)

Feature vector of (compute op, overlapping collective type):
    0 kernel class  1 base duration (ns)  2 collective type  3 largest message (bytes)
    4 most members  5 all-reduce algorithm  6 intra-server bandwidth  7 inter-server
    bandwidth (MB/s)  8-11 the class's four kernel metrics
"""
from __future__ import annotations

import numpy as np

TREE_NODE_DTYPE = np.dtype([("feature", "<i4"), ("left", "<i4"), ("right", "<i4"), ("value", "<i4"),
                            ("threshold", "<i8")])
N_FEATURES = 12
MAX_DEPTH = 12


def _threshold(rng, f):
    if f == 0:
        return int(rng.integers(1, 8))                     # kernel class
    if f == 1:
        return int(np.rint(50_000 * np.exp(0.7 * rng.standard_normal())))   # duration, ns
    if f == 2:
        return int(rng.integers(1, 4))                     # collective type
    if f == 3:
        return int(2 ** rng.uniform(16, 29))               # message bytes
    if f == 4:
        return int(rng.integers(2, 65))                    # members
    if f == 5:
        return 1                                           # ring / tree
    if f in (6, 7):
        return int(rng.integers(20_000, 400_001))          # bandwidths
    return int(rng.integers(100, 1000))                    # per-mille metrics


class _Builder:
    def __init__(self):
        self.rows = []

    def leaf(self, value):
        self.rows.append((-1, 0, 0, int(value), 0))
        return len(self.rows) - 1

    def split(self, feature, threshold):
        self.rows.append([feature, -1, -1, 0, int(threshold)])
        return len(self.rows) - 1

    def link(self, i, left, right):
        self.rows[i][1], self.rows[i][2] = left, right

    def array(self):
        out = np.zeros(len(self.rows), TREE_NODE_DTYPE)
        for i, r in enumerate(self.rows):
            out[i] = tuple(r)
        return out


def synthetic_forest(seed: int, n_trees: int = 64, max_depth: int = MAX_DEPTH, base: int = 72090,
                     leaf_mean: float = 250.0, leaf_sd: float = 900.0) -> dict:
    """n_trees random trees; a node at depth d splits with probability 0.9, 0.65 or 0.4
    (d < 4, d < 8, else) until max_depth; leaves draw N(leaf_mean, leaf_sd) Q16 units
    (base 72090 = 1.1; 64 trees add about +0.24 on average)."""
    rng = np.random.default_rng(seed)
    b = _Builder()
    roots = []

    def grow(depth):
        p = 0.9 if depth < 4 else 0.65 if depth < 8 else 0.4
        if depth >= max_depth or rng.random() > p:
            return b.leaf(np.rint(rng.normal(leaf_mean, leaf_sd)))
        f = int(rng.integers(0, N_FEATURES))
        i = b.split(f, _threshold(rng, f))
        left = grow(depth + 1)
        right = grow(depth + 1)
        b.link(i, left, right)
        return i

    for _ in range(n_trees):
        roots.append(grow(0))
    metrics = rng.integers(100, 1000, (8, 4)).astype(np.int64)
    return {"nodes": b.array(), "roots": np.array(roots, np.int32), "base": int(base), "class_metrics": metrics}


def table_forest(table) -> dict:
    """One tree that predicts table[class][type] exactly (splits on class, then type):
    base 65536, leaf value table[k][t] - 65536."""
    table = np.asarray(table, np.int64).reshape(8, 4)
    b = _Builder()

    def over(lo, hi, feature, leaf_of):
        if hi - lo == 1:
            return leaf_of(lo)
        mid = (lo + hi) // 2
        i = b.split(feature, mid)
        left = over(lo, mid, feature, leaf_of)
        right = over(mid, hi, feature, leaf_of)
        b.link(i, left, right)
        return i

    root = over(0, 8, 0, lambda k: over(0, 4, 2, lambda t: b.leaf(table[k][t] - 65536)))
    return {"nodes": b.array(), "roots": np.array([root], np.int32), "base": 65536,
            "class_metrics": np.zeros((8, 4), np.int64)}
