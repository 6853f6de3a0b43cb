"""Rows in compressed sparse row form, written from the definition -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this module; the library never does and shares no code with it.

Row i holds values[indptr[i]:indptr[i+1]] at features indices[same range]; every other
feature is 0.0.  Indices outside [0, n_features) are ignored; indices within a row are
distinct.
"""
from __future__ import annotations

import numpy as np


def densify(indptr, indices, values, n_rows: int, n_features: int) -> np.ndarray:
    X = np.zeros((n_rows, n_features), np.float32)
    indptr = np.asarray(indptr, np.int64)
    for i in range(n_rows):
        for e in range(indptr[i], indptr[i + 1]):
            f = int(indices[e])
            if 0 <= f < n_features:
                X[i, f] = values[e]
    return X
