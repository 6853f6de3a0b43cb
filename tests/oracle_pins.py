"""Pins for the CPU oracle: facts fixed by the mathematics, not by the oracle's code.

Each ``pin_*`` function takes an oracle library handle (``oracle.load(path)``) and
raises AssertionError on a mismatch.  ``test_oracle_pins.py`` runs them against the
real oracle and against deliberately broken copies of it (a flipped tie rule, a
swapped child, a dropped tree, ...), each of which must fail at least one pin.
"""
from __future__ import annotations

import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np

import oracle
from synth import (AGG_MEAN, AGG_SUM, XFORM_IDENTITY, XFORM_SIGMOID, XFORM_SOFTMAX, CONFIGS,
                   concat_trees, make_workload, perfect_tree_arrays, random_tiny_forest)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "w1_w2.txt")
F32 = np.float32


# ------------------------------------------------------------------ helpers
def _tree(nodes, leaves, n):
    """nodes: {id: (f, t, l, r)}, leaves: {id: value} -> per-tree arrays."""
    feat = np.full(n, -1, np.int32)
    thr = np.zeros(n, np.float32)
    l = np.full(n, -1, np.int32)
    r = np.full(n, -1, np.int32)
    v = np.zeros(n, np.float32)
    for i, (f, t, a, b) in nodes.items():
        feat[i], thr[i], l[i], r[i] = f, t, a, b
    for i, val in leaves.items():
        v[i] = val
    return feat, thr, l, r, v


def w1():
    return _tree({0: (0, 0.5, 1, 2), 1: (1, 0.25, 3, 4), 2: (1, 0.75, 5, 6)},
                 {3: 1.0, 4: 2.0, 5: 3.0, 6: 4.0}, 7)


def stump():
    return _tree({0: (1, 0.5, 1, 2)}, {1: -1.0, 2: 1.0}, 3)


def const(c=0.5):
    return _tree({}, {0: c}, 1)


def read_golden():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        p = line.split()
        xs = [float.fromhex(s) if s.startswith(("0x", "-0x")) else float(s) for s in p[:2]]
        leaves = [int(s) for s in p[2:5]]
        total = Fraction(p[5])
        mean = Fraction(p[6])
        rows.append((xs, leaves, total, mean))
    return rows


def dec_exp(x: float) -> Decimal:
    getcontext().prec = 40
    return Decimal(x).exp()


def dec_sigmoid(z: float) -> float:
    """High-precision logistic function via the decimal module (independent of libm)."""
    getcontext().prec = 40
    return float(Decimal(1) / (Decimal(1) + dec_exp(-z)))


def dec_softmax(z):
    getcontext().prec = 40
    e = [dec_exp(float(v)) for v in z]
    s = sum(e, Decimal(0))
    return [float(v / s) for v in e]


def run(lib, forest, X, leaves=True):
    return oracle.predict(forest, np.asarray(X, np.float32), want_leaves=leaves, lib=lib)


# -------------------------------------------------------------------- pins
def pin_hand_worked(lib):
    """P1: the hand-worked depth-2 tree W1 and the ensemble W2 = [W1, stump, constant]."""
    rows = read_golden()
    X = np.array([r[0] for r in rows], np.float32)
    f_sum = concat_trees([w1(), stump(), const()], 2, aggregate=AGG_SUM)
    out, lv, visits = run(lib, f_sum, X)
    for i, (_, leaves, total, mean) in enumerate(rows):
        assert list(lv[i]) == leaves, (i, list(lv[i]), leaves)
        assert out[i, 0] == float(total), (i, out[i, 0], total)
    assert visits == len(rows) * (2 + 1 + 0)
    f_mean = concat_trees([w1(), stump(), const()], 2, aggregate=AGG_MEAN)
    out, _, _ = run(lib, f_mean, X)
    for i, (_, _, total, mean) in enumerate(rows):
        assert abs(out[i, 0] - float(mean)) <= 1e-15 * abs(float(mean)), (i, out[i, 0], mean)
    f_sig = concat_trees([w1(), stump(), const()], 2, aggregate=AGG_SUM, transform=XFORM_SIGMOID)
    out, _, _ = run(lib, f_sig, X)
    for i, (_, _, total, _) in enumerate(rows):
        want = dec_sigmoid(float(total))
        assert abs(out[i, 0] - want) <= 1e-15, (i, out[i, 0], want)
    # two classes: W1 -> class 0, stump -> class 1
    f_sm = concat_trees([w1(), stump()], 2, n_classes=2, tree_class=[0, 1], transform=XFORM_SOFTMAX)
    out, _, _ = run(lib, f_sm, X)
    for i, (_, leaves, _, _) in enumerate(rows):
        z = [{3: 1.0, 4: 2.0, 5: 3.0, 6: 4.0}[leaves[0]], {1: -1.0, 2: 1.0}[leaves[1]]]
        want = dec_softmax(z)
        assert max(abs(a - b) for a, b in zip(out[i], want)) <= 1e-15, (i, out[i], want)


def _leaf_boxes(feat, thr, l, r, n_features):
    """Each leaf's region: per feature an interval (lo, hi] for numbers, and whether NaN
    may take that feature (only if the path never goes left on it)."""
    boxes = {}
    stack = [(0, [(-math.inf, math.inf, True) for _ in range(n_features)])]
    while stack:
        n, box = stack.pop()
        if l[n] == -1:
            boxes[n] = box
            continue
        f, t = int(feat[n]), float(thr[n])
        lo, hi, nan_ok = box[f]
        bl = list(box)
        bl[f] = (lo, min(hi, t), False)          # x <= t
        br = list(box)
        br[f] = (max(lo, t), hi, nan_ok)         # x > t, or NaN
        stack.append((int(l[n]), bl))
        stack.append((int(r[n]), br))
    return boxes


def _in_box(x, box):
    for v, (lo, hi, nan_ok) in zip(x, box):
        if math.isnan(v):
            if not nan_ok:
                return False
        elif not (lo < v <= hi) and not (v == -math.inf and lo == -math.inf and v <= hi):
            return False
    return True


def pin_leaf_regions(lib, n_forests=12, seed=11):
    """P2: brute force over every leaf region of tiny trees, probing each threshold,
    its float neighbours, +-0, +-inf and NaN."""
    rng = np.random.default_rng(seed)
    grid = np.array([-1.5, -0.25, 0.0, 0.25, 1.0, 2.0], np.float32)
    for i in range(n_forests):
        F = 2 + i % 2
        f = random_tiny_forest(rng, 1, F, max_depth=4, p_split=0.8, thr_grid=grid)
        feat, thr, l, r, v = f.tree(0)
        boxes = _leaf_boxes(feat, thr, l, r, F)
        cand = {0.0, -0.0, math.inf, -math.inf, math.nan}
        for t in thr[l >= 0]:
            t = F32(t)
            cand |= {float(t), float(np.nextafter(t, F32(np.inf))), float(np.nextafter(t, F32(-np.inf)))}
        cand = sorted(cand, key=lambda c: (math.isnan(c), c))
        pts = np.array(np.meshgrid(*[cand] * F, indexing="ij")).reshape(F, -1).T.astype(np.float32)
        _, lv, _ = run(lib, f, pts)
        for p, leaf in zip(pts, lv[:, 0]):
            inside = [n for n, b in boxes.items() if _in_box([float(x) for x in p], b)]
            assert inside == [int(leaf)], (i, p, inside, int(leaf))


def pin_closed_forms(lib):
    """P3: special cases that reduce to library routines or exact values."""
    rng = np.random.default_rng(5)
    X = rng.standard_normal((4000, 6)).astype(np.float32)
    X[rng.random(X.shape) < 0.02] = np.nan
    X[:50, 3] = np.float32(0.125)                         # exact ties
    # a stump is numpy.where on one column
    f = concat_trees([_tree({0: (3, 0.125, 1, 2)}, {1: -2.5, 2: 7.0}, 3)], 6)
    out, lv, vis = run(lib, f, X)
    want = np.where(X[:, 3] <= F32(0.125), -2.5, 7.0)
    assert np.array_equal(out[:, 0], want)
    assert vis == X.shape[0]
    # an oblivious perfect tree (level d splits on (f_d, t_d) everywhere): leaf id in closed form
    D = 4
    fd = rng.integers(0, 6, D)
    td = rng.standard_normal(D).astype(np.float32)
    n_int = (1 << D) - 1
    depth_of = np.floor(np.log2(np.arange(n_int) + 1)).astype(int)
    leaves = rng.standard_normal(1 << D).astype(np.float32)
    f = concat_trees([perfect_tree_arrays(D, fd[depth_of], td[depth_of], leaves)], 6)
    out, lv, vis = run(lib, f, X)
    bits = [(~(X[:, fd[d]] <= td[d])).astype(np.int64) for d in range(D)]
    want_leaf = (1 << D) - 1 + sum(b << (D - 1 - d) for d, b in enumerate(bits))
    assert np.array_equal(lv[:, 0], want_leaf)
    assert np.array_equal(out[:, 0], leaves[want_leaf - n_int].astype(np.float64))
    assert vis == X.shape[0] * D
    # a depth-0 tree returns its constant and visits nothing
    f = concat_trees([const(-3.25)], 6)
    out, lv, vis = run(lib, f, X)
    assert np.all(out[:, 0] == -3.25) and np.all(lv == 0) and vis == 0
    # the mean of T identical trees (dyadic leaves) is the tree itself
    t1 = perfect_tree_arrays(3, np.array([0, 1, 2, 3, 4, 5, 0]), np.zeros(7, np.float32),
                             np.arange(-4, 4) / 8.0)
    f1 = concat_trees([t1], 6)
    f7 = concat_trees([t1] * 7, 6, aggregate=AGG_MEAN)
    a, _, _ = run(lib, f1, X)
    b, _, _ = run(lib, f7, X)
    assert np.array_equal(a, b)
    # a base score is added once (sum) and outside the mean
    f = concat_trees([t1] * 3, 6, base_score=[0.75])
    c, _, _ = run(lib, f, X)
    assert np.array_equal(c, 3 * a + 0.75)
    f = concat_trees([t1] * 4, 6, aggregate=AGG_MEAN, base_score=[0.75])
    c, _, _ = run(lib, f, X)
    assert np.array_equal(c, a + 0.75)
    # sigmoid(0) = 1/2 exactly; sigmoid(z) + sigmoid(-z) = 1
    f = concat_trees([const(0.0)], 6, transform=XFORM_SIGMOID)
    c, _, _ = run(lib, f, X[:3])
    assert np.all(c == 0.5)
    for z in (0.5, 3.0, 17.0, -40.0):
        fp = concat_trees([const(z)], 6, transform=XFORM_SIGMOID)
        fn = concat_trees([const(-z)], 6, transform=XFORM_SIGMOID)
        p, _, _ = run(lib, fp, X[:1])
        q, _, _ = run(lib, fn, X[:1])
        assert abs(p[0, 0] + q[0, 0] - 1.0) <= 1e-15
        assert abs(p[0, 0] - dec_sigmoid(z)) <= 1e-16 + 1e-15 * dec_sigmoid(z)
    # softmax of equal logits is uniform; softmax of two classes is a sigmoid of the gap
    f = concat_trees([const(1.5)] * 4, 6, n_classes=4, transform=XFORM_SOFTMAX)
    c, _, _ = run(lib, f, X[:2])
    assert np.all(c == 0.25)
    f = concat_trees([const(2.0), const(-1.0), const(0.5)], 6, n_classes=3, tree_class=[2, 0, 1],
                     transform=XFORM_SOFTMAX)
    c, _, _ = run(lib, f, X[:1])
    want = dec_softmax([-1.0, 0.5, 2.0])
    assert max(abs(a - b) for a, b in zip(c[0], want)) <= 1e-16


def pin_invariants(lib, seed=3):
    """P4: one leaf per (row, tree), the path agrees with every compare, visits = sum of depths."""
    rng = np.random.default_rng(seed)
    f = random_tiny_forest(rng, 25, 5, max_depth=7, p_split=0.75,
                           thr_grid=np.array([-1, -0.5, 0, 0.5, 1], np.float32))
    X = rng.standard_normal((700, 5)).astype(np.float32)
    X[:, 2] = np.round(X[:, 2] * 2) / 2                   # many exact ties on feature 2
    X[5, :] = np.nan
    _, lv, vis = run(lib, f, X)
    total_depth = 0
    for t in range(f.n_trees):
        feat, thr, l, r, _ = f.tree(t)
        parent = {int(c): (p, side) for p in range(len(l)) for side, c in ((0, l[p]), (1, r[p])) if c >= 0}
        hist = np.bincount(lv[:, t], minlength=len(l))
        assert hist.sum() == X.shape[0]
        assert np.all(hist[l >= 0] == 0)                  # only leaves are reached
        for i in range(X.shape[0]):
            n = int(lv[i, t])
            d = 0
            while n != 0:
                p, side = parent[n]
                went_left = bool(X[i, feat[p]] <= thr[p])
                assert went_left == (side == 0)
                n = p
                d += 1
            total_depth += d
    assert vis == total_depth


def numpy_traverse(forest, X):
    """Independent vectorized traversal (level-synchronous over all rows), with sums taken
    in ascending tree order in float64.  Returns (z before the transform, leaves)."""
    n = X.shape[0]
    K = forest.n_classes
    T = forest.n_trees
    tc = forest.tree_class if forest.tree_class is not None else np.arange(T) % K
    z = np.zeros((n, K))
    if forest.aggregate == AGG_SUM and forest.base_score is not None:
        z += forest.base_score.astype(np.float64)
    leaves = np.empty((n, T), np.int32)
    rows = np.arange(n)
    for t in range(T):
        feat, thr, l, r, v = forest.tree(t)
        node = np.zeros(n, np.int64)
        active = l[node] >= 0
        while active.any():
            idx = node[active]
            go_left = X[rows[active], feat[idx]] <= thr[idx]
            node[active] = np.where(go_left, l[idx], r[idx])
            active = l[node] >= 0
        leaves[:, t] = node
        z[:, tc[t]] = z[:, tc[t]] + v[node].astype(np.float64)
    if forest.aggregate == AGG_MEAN:
        cnt = np.bincount(tc, minlength=K).astype(np.float64)
        base = 0.0 if forest.base_score is None else forest.base_score.astype(np.float64)
        z = base + z / cnt
    return z, leaves


def pin_vectorized_crosscheck(lib, rows_per_config=(256, 128, 128, 24, 24)):
    """P5: the five workloads (row prefixes) against the independent vectorized traversal."""
    for name, nr in zip(CONFIGS, rows_per_config):
        w = make_workload(name, nr)
        X = w.X()
        out, lv, _ = run(lib, w.forest, X)
        z, lv2 = numpy_traverse(w.forest, X)
        assert np.array_equal(lv, lv2), name
        if w.forest.transform == XFORM_IDENTITY:
            assert np.array_equal(out, z), name
        elif w.forest.transform == XFORM_SIGMOID:
            want = np.array([dec_sigmoid(float(v)) for v in z[:, 0]])
            assert np.max(np.abs(out[:, 0] - want)) <= 1e-15, name
        else:
            want = np.array([dec_softmax(list(r)) for r in z])
            assert np.max(np.abs(out - want)) <= 1e-15, name


def pin_summation(lib, seed=9):
    """P6: dyadic leaves sum exactly in any order; general leaves stay within the
    sequential-summation error bound of the exact (fsum) result."""
    rng = np.random.default_rng(seed)
    f = random_tiny_forest(rng, 200, 4, max_depth=5, p_split=0.8, leaf_dyadic=True)
    X = rng.standard_normal((300, 4)).astype(np.float32)
    out, lv, _ = run(lib, f, X)
    vals = [f.value[f.tree_offsets[t]:f.tree_offsets[t + 1]] for t in range(f.n_trees)]
    for i in range(X.shape[0]):
        exact = math.fsum(float(vals[t][lv[i, t]]) for t in range(f.n_trees))
        assert out[i, 0] == exact
    f = random_tiny_forest(rng, 300, 4, max_depth=5, p_split=0.8)
    out, lv, _ = run(lib, f, X)
    vals = [f.value[f.tree_offsets[t]:f.tree_offsets[t + 1]] for t in range(f.n_trees)]
    eps = 2.0 ** -53
    for i in range(X.shape[0]):
        terms = [float(vals[t][lv[i, t]]) for t in range(f.n_trees)]
        exact = math.fsum(terms)
        bound = (len(terms) - 1) * eps * sum(abs(x) for x in terms) * 1.01
        assert abs(out[i, 0] - exact) <= bound


def pin_class_map(lib, seed=13):
    """Multiclass: class(t) = t mod K when no map is given; an explicit map routes trees."""
    rng = np.random.default_rng(seed)
    trees = [const(float(v)) for v in (rng.integers(-8, 8, 12) / 4.0)]
    X = np.zeros((2, 3), np.float32)
    f = concat_trees(trees, 3, n_classes=3)
    out, _, _ = run(lib, f, X)
    cv = [float(t[4][0]) for t in trees]
    want = [sum(cv[k::3]) for k in range(3)]
    assert np.array_equal(out[0], want)
    tcm = rng.integers(0, 3, 12)
    f = concat_trees(trees, 3, n_classes=3, tree_class=tcm, aggregate=AGG_MEAN)
    out, _, _ = run(lib, f, X)
    for k in range(3):
        sel = [cv[t] for t in range(12) if tcm[t] == k]
        assert out[0, k] == (sum(sel) / len(sel) if sel else out[0, k])


def pin_row_stride(lib, seed=17):
    """Each row reads its own features: permuting rows permutes the outputs."""
    rng = np.random.default_rng(seed)
    f = random_tiny_forest(rng, 10, 7, max_depth=6, p_split=0.8)
    X = rng.standard_normal((64, 7)).astype(np.float32)
    perm = rng.permutation(64)
    a, la, _ = run(lib, f, X)
    b, lb, _ = run(lib, f, X[perm])
    assert np.array_equal(a[perm], b) and np.array_equal(la[perm], lb)
    # and a single row evaluated alone gives the same answer
    c, lc, _ = run(lib, f, X[7:8])
    assert np.array_equal(c[0], a[7]) and np.array_equal(lc[0], la[7])


ALL_PINS = [pin_hand_worked, pin_leaf_regions, pin_closed_forms, pin_invariants,
            pin_vectorized_crosscheck, pin_summation, pin_class_map, pin_row_stride]
