"""Seeded synthetic forests and feature matrices.

Workloads are stand-ins for the tabular data of the paper's evaluation (Sec. 5.3
uses a public 51,630 x 90 regression set, which is not available here).  Every
input is synthetic and reproducible from its seed:

* X is generated in blocks of ``BLOCK_ROWS`` rows; block ``b`` comes from
  ``numpy.random.default_rng([seed, 1, b])``, so any block (hence any row) can be
  regenerated on its own, and a smaller problem is a prefix of the full one.
* Forest draws come from ``default_rng([seed, 2])`` and never depend on the row
  count: thresholds sampled "from the feature's column" are taken from the rows
  of block 0 (the first BLOCK_ROWS rows, always generated in full).
* Nodes are numbered breadth-first inside each tree, root = tree-local 0, a leaf
  has left == right == -1; ``permute_nodes`` renumbers nodes to exercise
  arbitrary caller numberings.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

AGG_SUM, AGG_MEAN = 0, 1
XFORM_IDENTITY, XFORM_SIGMOID, XFORM_SOFTMAX = 0, 1, 2

BLOCK_ROWS = 65536


@dataclass
class Forest:
    """Forest in the caller-facing array format (one entry per node, trees concatenated)."""
    n_features: int
    n_classes: int
    tree_offsets: np.ndarray          # int64 [T+1]
    feature: np.ndarray               # int32 [N]; ignored at leaves
    threshold: np.ndarray             # float32 [N]; ignored at leaves
    left: np.ndarray                  # int32 [N]; tree-local child id or -1
    right: np.ndarray                 # int32 [N]
    value: np.ndarray                 # float32 [N]; used at leaves
    tree_class: Optional[np.ndarray] = None   # int32 [T] or None (class t mod K)
    aggregate: int = AGG_SUM
    transform: int = XFORM_IDENTITY
    base_score: Optional[np.ndarray] = None    # float32 [K] or None (zeros)

    @property
    def n_trees(self) -> int:
        return int(self.tree_offsets.shape[0] - 1)

    @property
    def n_nodes(self) -> int:
        return int(self.tree_offsets[-1])

    def tree(self, t: int):
        a, b = int(self.tree_offsets[t]), int(self.tree_offsets[t + 1])
        return (self.feature[a:b], self.threshold[a:b], self.left[a:b], self.right[a:b], self.value[a:b])


@dataclass
class Workload:
    name: str
    seed: int
    n_rows: int
    n_features: int
    x_kind: str                       # "uniform" | "normal" | "sparse_uniform"
    forest: Forest
    description: str = ""
    x_params: dict = field(default_factory=dict)

    def X(self, n_rows: Optional[int] = None) -> np.ndarray:
        n = self.n_rows if n_rows is None else n_rows
        return x_rows(self.seed, self.x_kind, self.n_features, 0, n, **self.x_params)


# ----------------------------------------------------------------------------- X
def x_block(seed: int, kind: str, n_features: int, b: int, keep_prob: float = 0.2) -> np.ndarray:
    """Block ``b`` of the feature matrix: BLOCK_ROWS x n_features float32, row-major."""
    rng = np.random.default_rng([seed, 1, b])
    shape = (BLOCK_ROWS, n_features)
    if kind == "uniform":
        return rng.random(shape, dtype=np.float32)
    if kind == "normal":
        return rng.standard_normal(shape, dtype=np.float32)
    if kind == "sparse_uniform":
        v = rng.random(shape, dtype=np.float32)
        keep = rng.random(shape, dtype=np.float32) < np.float32(keep_prob)
        return np.where(keep, v, np.float32(0.0)).astype(np.float32)
    raise ValueError(kind)


def x_rows(seed: int, kind: str, n_features: int, r0: int, r1: int, **kw) -> np.ndarray:
    """Rows [r0, r1) of the feature matrix (float32, C-contiguous)."""
    out = np.empty((max(r1 - r0, 0), n_features), dtype=np.float32)
    r = r0
    while r < r1:
        b = r // BLOCK_ROWS
        lo = r - b * BLOCK_ROWS
        hi = min(BLOCK_ROWS, r1 - b * BLOCK_ROWS)
        out[r - r0:r - r0 + hi - lo] = x_block(seed, kind, n_features, b, **kw)[lo:hi]
        r += hi - lo
    return out


def x_rows_threaded(seed: int, kind: str, n_features: int, r0: int, r1: int, threads: int = 8,
                    **kw) -> np.ndarray:
    """Rows [r0, r1) as ``x_rows``, the blocks drawn on ``threads`` threads (each block has its
    own generator, so the result does not depend on the thread count)."""
    from concurrent.futures import ThreadPoolExecutor
    out = np.empty((max(r1 - r0, 0), n_features), dtype=np.float32)
    if r1 <= r0:
        return out
    spans = []
    r = r0
    while r < r1:
        e = min(r1, (r // BLOCK_ROWS + 1) * BLOCK_ROWS)
        spans.append((r, e))
        r = e

    def fill(span):
        a, b = span
        out[a - r0:b - r0] = x_rows(seed, kind, n_features, a, b, **kw)

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(fill, spans))
    return out


def x_take(seed: int, kind: str, n_features: int, rows, **kw) -> np.ndarray:
    """The given rows (any order) of the feature matrix, generating each needed block once."""
    rows = np.asarray(rows, np.int64)
    out = np.empty((rows.shape[0], n_features), dtype=np.float32)
    blocks = rows // BLOCK_ROWS
    for b in np.unique(blocks):
        sel = np.nonzero(blocks == b)[0]
        out[sel] = x_block(seed, kind, n_features, int(b), **kw)[rows[sel] - b * BLOCK_ROWS]
    return out


# ------------------------------------------------------------------------- trees
def perfect_tree_arrays(depth: int, feats: np.ndarray, thrs: np.ndarray, leaves: np.ndarray):
    """Arrays of one perfect tree in breadth-first numbering.

    feats/thrs: the 2^depth - 1 internal nodes in BFS order; leaves: the 2^depth leaf values."""
    n_int = (1 << depth) - 1
    n = (1 << (depth + 1)) - 1
    feature = np.full(n, -1, np.int32)
    threshold = np.zeros(n, np.float32)
    left = np.full(n, -1, np.int32)
    right = np.full(n, -1, np.int32)
    value = np.zeros(n, np.float32)
    idx = np.arange(n_int)
    feature[:n_int] = feats
    threshold[:n_int] = thrs
    left[:n_int] = 2 * idx + 1
    right[:n_int] = 2 * idx + 2
    value[n_int:] = leaves
    return feature, threshold, left, right, value


def ragged_tree_structure(rng: np.random.Generator, p_split: float, max_depth: int):
    """Grow one tree: every node above max_depth splits with probability p_split.

    Returns (left, right, depth) in breadth-first numbering; children of a node are
    numbered consecutively (right = left + 1)."""
    left = [-1]
    right = [-1]
    depth = [0]
    frontier = [0]
    d = 0
    while frontier and d < max_depth:
        split = rng.random(len(frontier)) < p_split
        nxt = []
        for node, s in zip(frontier, split):
            if s:
                l = len(left)
                left[node] = l
                right[node] = l + 1
                left += [-1, -1]
                right += [-1, -1]
                depth += [d + 1, d + 1]
                nxt += [l, l + 1]
        frontier = nxt
        d += 1
    return np.asarray(left, np.int32), np.asarray(right, np.int32), np.asarray(depth, np.int32)


def concat_trees(trees, n_features, n_classes=1, tree_class=None, aggregate=AGG_SUM,
                 transform=XFORM_IDENTITY, base_score=None) -> Forest:
    """Build a Forest from a list of per-tree (feature, threshold, left, right, value) arrays."""
    sizes = [len(t[0]) for t in trees]
    offs = np.zeros(len(trees) + 1, np.int64)
    offs[1:] = np.cumsum(sizes)
    cat = [np.concatenate([t[i] for t in trees]) if trees else np.zeros(0) for i in range(5)]
    return Forest(
        n_features=n_features, n_classes=n_classes, tree_offsets=offs,
        feature=cat[0].astype(np.int32), threshold=cat[1].astype(np.float32),
        left=cat[2].astype(np.int32), right=cat[3].astype(np.int32), value=cat[4].astype(np.float32),
        tree_class=None if tree_class is None else np.asarray(tree_class, np.int32),
        aggregate=aggregate, transform=transform,
        base_score=None if base_score is None else np.asarray(base_score, np.float32))


def permute_nodes(f: Forest, rng: np.random.Generator) -> Forest:
    """Renumber the non-root nodes of every tree at random (the root stays tree-local 0)."""
    trees = []
    for t in range(f.n_trees):
        feat, thr, l, r, v = f.tree(t)
        n = len(feat)
        perm = np.concatenate([[0], 1 + rng.permutation(n - 1)]).astype(np.int64)  # old -> new
        inv = np.empty(n, np.int64)
        inv[perm] = np.arange(n)
        def remap(c):
            c = c.astype(np.int64)
            out = np.where(c >= 0, perm[np.maximum(c, 0)], -1)
            return out[inv].astype(np.int32)
        trees.append((feat[inv], thr[inv], remap(l), remap(r), v[inv]))
    return concat_trees(trees, f.n_features, f.n_classes, f.tree_class, f.aggregate, f.transform,
                        f.base_score)


def random_tiny_forest(rng: np.random.Generator, n_trees: int, n_features: int, max_depth: int,
                       p_split: float = 0.7, thr_grid=None, leaf_dyadic: bool = False,
                       n_classes: int = 1, aggregate=AGG_SUM, transform=XFORM_IDENTITY) -> Forest:
    """Small random ragged forest; thresholds from ``thr_grid`` (ties likely) or N(0,1)."""
    trees = []
    for _ in range(n_trees):
        l, r, _d = ragged_tree_structure(rng, p_split, max_depth)
        n = len(l)
        feat = rng.integers(0, n_features, n).astype(np.int32)
        if thr_grid is not None:
            thr = np.asarray(thr_grid, np.float32)[rng.integers(0, len(thr_grid), n)]
        else:
            thr = rng.standard_normal(n).astype(np.float32)
        if leaf_dyadic:
            val = (rng.integers(-2048, 2049, n) / 256.0).astype(np.float32)
        else:
            val = rng.standard_normal(n).astype(np.float32)
        leaf = l < 0
        feat[leaf] = -1
        thr[leaf] = 0.0
        val[~leaf] = 0.0
        trees.append((feat, thr, l, r, val))
    return concat_trees(trees, n_features, n_classes, None, aggregate, transform)


def with_vector_leaves(f: Forest, n_classes: int, rng: np.random.Generator,
                       aggregate=AGG_MEAN, transform=XFORM_IDENTITY) -> Forest:
    """The same trees with a class-probability vector in every leaf (a tree classifier's
    leaves: random class counts, normalised), ``value`` of shape [N, n_classes] (zeros at
    internal nodes).  Every tree votes in every class."""
    leaf = f.left < 0
    counts = rng.integers(0, 20, (f.n_nodes, n_classes)).astype(np.float64)
    counts[leaf & (counts.sum(1) == 0), 0] = 1.0
    v = np.zeros((f.n_nodes, n_classes), np.float32)
    v[leaf] = (counts[leaf] / counts[leaf].sum(1, keepdims=True)).astype(np.float32)
    return Forest(n_features=f.n_features, n_classes=n_classes, tree_offsets=f.tree_offsets,
                  feature=f.feature, threshold=f.threshold, left=f.left, right=f.right, value=v,
                  tree_class=None, aggregate=aggregate, transform=transform, base_score=None)


# ------------------------------------------------------------------- workloads
def _threshold_pool(seed, kind, n_features, x_params):
    return x_block(seed, kind, n_features, 0, **x_params)


def make_forest(spec: dict) -> Forest:
    seed = spec["seed"]
    F = spec["n_features"]
    rng = np.random.default_rng([seed, 2])
    pool = None
    if spec["thr"] == "column":
        pool = _threshold_pool(seed, spec["x"], F, spec.get("x_params", {}))
    trees = []
    T = spec["n_trees"]
    for t in range(T):
        if spec["shape"] == "perfect":
            D = spec["depth"]
            n_int = (1 << D) - 1
            feats = rng.integers(0, F, n_int).astype(np.int32)
            if spec["thr"] == "uniform":
                thrs = rng.random(n_int, dtype=np.float32)
            else:
                rows = rng.integers(0, pool.shape[0], n_int)
                thrs = pool[rows, feats]
            leaves = (rng.standard_normal(1 << D) * spec["leaf_sigma"]).astype(np.float32)
            trees.append(perfect_tree_arrays(D, feats, thrs, leaves))
        else:
            l, r, _d = ragged_tree_structure(rng, spec["p_split"], spec["max_depth"])
            n = len(l)
            internal = l >= 0
            feat = np.full(n, -1, np.int32)
            thr = np.zeros(n, np.float32)
            val = np.zeros(n, np.float32)
            ni = int(internal.sum())
            feat[internal] = rng.integers(0, F, ni)
            rows = rng.integers(0, pool.shape[0], ni)
            thr[internal] = pool[rows, feat[internal]]
            val[~internal] = (rng.standard_normal(n - ni) * spec["leaf_sigma"]).astype(np.float32)
            trees.append((feat, thr, l, r, val))
    K = spec.get("n_classes", 1)
    tc = None
    if K > 1:
        tc = (np.arange(T) % K).astype(np.int32)
    return concat_trees(trees, F, K, tc, spec["agg"], spec["xform"],
                        np.zeros(K, np.float32) if spec.get("base") is not None else None)


CONFIGS = {
    "dt_d3": dict(
        seed=0, n_rows=10_000, n_features=28, x="uniform", shape="perfect", depth=3, n_trees=1,
        thr="uniform", leaf_sigma=1.0, agg=AGG_SUM, xform=XFORM_IDENTITY,
        description="single perfect decision tree, depth 3, 10,000 x 28 U[0,1) rows; output = leaf value"),
    "rf_d8": dict(
        seed=1, n_rows=1_000_000, n_features=28, x="normal", shape="perfect", depth=8, n_trees=100,
        thr="column", leaf_sigma=1.0, agg=AGG_MEAN, xform=XFORM_IDENTITY,
        description="random-forest regression, 100 perfect depth-8 trees, 1M x 28 N(0,1) rows; mean"),
    "gbdt_d6": dict(
        seed=2, n_rows=1_000_000, n_features=28, x="normal", shape="perfect", depth=6, n_trees=500,
        thr="column", leaf_sigma=0.1, agg=AGG_SUM, xform=XFORM_SIGMOID, base=0.0,
        description="binary GBDT, 500 perfect depth-6 trees, 1M x 28 N(0,1) rows; sigmoid(0 + sum)"),
    "mc_gbdt_d8": dict(
        seed=3, n_rows=100_000, n_features=784, x="sparse_uniform", x_params={"keep_prob": 0.2},
        shape="perfect", depth=8, n_trees=1000, n_classes=10, thr="column", leaf_sigma=0.1,
        agg=AGG_SUM, xform=XFORM_SOFTMAX,
        description="10-class GBDT, 1000 perfect depth-8 trees (class = t mod 10), 100k x 784 "
                    "U[0,1) rows with 80% zeros; softmax"),
    "ragged_d12": dict(
        seed=4, n_rows=4_000_000, n_features=256, x="normal", shape="ragged", p_split=0.85,
        max_depth=12, n_trees=1000, thr="column", leaf_sigma=1.0, agg=AGG_SUM, xform=XFORM_IDENTITY,
        description="1000 ragged trees (split prob 0.85, max depth 12), 4M x 256 N(0,1) rows; sum"),
}

# Extra workloads (not part of the five benchmark configurations): shallow forests to compare
# the matrix-multiply lowering with the traversal kernels, and a forest of ragged trees on
# narrow rows (the shape of a random-forest classifier's trees; with class-vector leaves via
# synth.with_vector_leaves) for the LDS-chunked ragged kernel.
EXTRA_CONFIGS = {
    "ragged_rf_28": dict(
        seed=13, n_rows=1_000_000, n_features=28, x="normal", shape="ragged", p_split=0.85,
        max_depth=12, n_trees=100, thr="column", leaf_sigma=1.0, agg=AGG_MEAN, xform=XFORM_IDENTITY,
        description="100 ragged trees (split prob 0.85, max depth 12), 1M x 28 N(0,1) rows; mean"),
    "shallow_d3": dict(
        seed=11, n_rows=1_000_000, n_features=28, x="normal", shape="perfect", depth=3, n_trees=100,
        thr="column", leaf_sigma=0.1, agg=AGG_SUM, xform=XFORM_SIGMOID, base=0.0,
        description="binary GBDT, 100 perfect depth-3 trees, 1M x 28 N(0,1) rows; sigmoid"),
    "shallow_d4": dict(
        seed=12, n_rows=1_000_000, n_features=28, x="normal", shape="perfect", depth=4, n_trees=50,
        thr="column", leaf_sigma=0.1, agg=AGG_SUM, xform=XFORM_SIGMOID, base=0.0,
        description="binary GBDT, 50 perfect depth-4 trees, 1M x 28 N(0,1) rows; sigmoid"),
}

_FOREST_CACHE: dict = {}


def make_workload(name: str, n_rows: Optional[int] = None) -> Workload:
    spec = CONFIGS[name] if name in CONFIGS else EXTRA_CONFIGS[name]
    if name not in _FOREST_CACHE:
        _FOREST_CACHE[name] = make_forest(spec)
    return Workload(name=name, seed=spec["seed"], n_rows=spec["n_rows"] if n_rows is None else n_rows,
                    n_features=spec["n_features"], x_kind=spec["x"], forest=_FOREST_CACHE[name],
                    description=spec["description"], x_params=spec.get("x_params", {}))
