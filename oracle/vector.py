"""Forests whose leaves hold one value per class -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this module; the library never does and shares no code with it.

Tree classifiers of the paper's CML suite (decision, extra and random forests of trees; its
evaluation names ExtraTreeClassifier) store a class-probability vector in every leaf, and a
forest of them averages the vectors of the leaves a row reaches (the aggregation category of
the classical operator representation, Sec. 3.2 and Sec. 4.2; Table 4's sum/mean).  Written
from that definition:

  leaf(r, t)  the leaf row r reaches in tree t (the scalar oracle's walk: left iff x <= t)
  acc[k]      = base[k] (SUM) or 0 (MEAN); then for t = 0, 1, ..., T-1 in turn
  acc[k]      = acc[k] + double(V[leaf(r, t), k])          (one double add per tree)
  z[k]        = acc[k] (SUM) or base[k] + acc[k] / T (MEAN: every tree votes in every class)
  out         = z, or softmax(z): m = max_k z[k], e[k] = exp(z[k] - m), s = e[0] + e[1] + ...
                in class order, out[k] = e[k] / s
The class of largest value (the first on ties) is the label.
"""
from __future__ import annotations

import numpy as np

from . import predict as _scalar_predict

AGG_SUM, AGG_MEAN = 0, 1
XFORM_IDENTITY, XFORM_SOFTMAX = 0, 2


def leaves(forest, X: np.ndarray, threads: int = 1, with_visits: bool = False):
    """Tree-local leaf ids [n, T] from the scalar oracle's walk (the leaf values play no part);
    with_visits: also the number of internal-node visits."""
    _, lv, visits = _scalar_predict(_as_scalar(forest), X, want_leaves=True, threads=threads)
    return (lv, visits) if with_visits else lv


def _as_scalar(forest):
    import dataclasses
    v = np.asarray(forest.value)
    if v.ndim == 1:
        return forest
    return dataclasses.replace(forest, value=np.ascontiguousarray(v[:, 0], np.float32),
                               n_classes=1, tree_class=None, transform=XFORM_IDENTITY,
                               base_score=None)


def predict(forest, X: np.ndarray, threads: int = 1, with_visits: bool = False):
    """(out float64 [n, K], leaves int32 [n, T]) for a forest whose ``value`` is [N, K]; with
    with_visits, also the number of internal-node visits."""
    V = np.asarray(forest.value, np.float32)
    assert V.ndim == 2, "value must hold one row of class values per node"
    K = V.shape[1]
    T = int(forest.n_trees)
    lv, visits = leaves(forest, X, threads, with_visits=True)
    n = lv.shape[0]
    base = np.zeros(K) if forest.base_score is None else np.asarray(forest.base_score, np.float64)
    acc = np.tile(base, (n, 1)) if forest.aggregate == AGG_SUM else np.zeros((n, K))
    offs = np.asarray(forest.tree_offsets, np.int64)
    for t in range(T):
        acc = acc + V[offs[t] + lv[:, t].astype(np.int64)].astype(np.float64)
    z = acc if forest.aggregate == AGG_SUM else base[None, :] + acc / float(T)
    if forest.transform == XFORM_SOFTMAX:
        m = z.max(axis=1, keepdims=True)
        e = np.exp(z - m)
        s = np.zeros(n)
        for k in range(K):
            s = s + e[:, k]
        z = e / s[:, None]
    elif forest.transform != XFORM_IDENTITY:
        raise ValueError("vector leaves take the identity or softmax link")
    return (z, lv, visits) if with_visits else (z, lv)


def labels(out: np.ndarray) -> np.ndarray:
    """The first class of largest value."""
    return np.argmax(out, axis=1).astype(np.int32)
