"""Exact feature quantization, written from its definition -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this module; the library never does and shares no code with it.

Definition (the "data type rewriting" of the paper's Table 2 applied to the inputs, as the
build plan reads it): for feature f, let U_f be the forest's distinct split thresholds on f
(internal nodes only; -0.0 and +0.0 count as one value).  The bin of a value x is
#{u in U_f : u < x}; a NaN gets |U_f|.  A threshold t in U_f has rank k = #{u in U_f : u < t},
and x <= t exactly when bin(x) <= k (NaN: false on both sides), so a walk on bins reaches
the same leaves as the walk on fp32 values.
"""
from __future__ import annotations

import numpy as np


def tables(forest):
    """Per feature, the sorted distinct thresholds as float32 arrays (-0 stored as +0)."""
    internal = forest.left >= 0
    feat = forest.feature[internal]
    thr = forest.threshold[internal].astype(np.float32) + np.float32(0.0)  # -0 + 0 = +0
    out = []
    for f in range(forest.n_features):
        out.append(np.unique(thr[feat == f]).astype(np.float32))
    return out


def bin_width(tabs) -> int:
    """Bytes per bin: 1 if every feature has at most 255 thresholds, 2 if at most 65535."""
    m = max((len(u) for u in tabs), default=0)
    return 1 if m <= 255 else (2 if m <= 65535 else 0)


def bin_rows(tabs, X: np.ndarray) -> np.ndarray:
    """bin(x) for every element of X [n, F] (int64)."""
    X = np.asarray(X, np.float32)
    out = np.empty(X.shape, np.int64)
    for f, u in enumerate(tabs):
        col = X[:, f]
        b = np.searchsorted(u, col, side="left")   # number of table entries strictly below
        b[np.isnan(col)] = len(u)
        out[:, f] = b
    return out


def rank(tabs, f: int, t: float) -> int:
    """Rank of threshold t among feature f's distinct thresholds."""
    return int(np.searchsorted(tabs[f], np.float32(t) + np.float32(0.0), side="left"))
