"""Preprocessing ahead of the forest, written from its definition -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this module; the library never does and shares no code with it.

The scalers of the paper's CML suite (its evaluation names Binarizer, Normalizer,
MinMaxScaler and RobustScaler; StandardScaler is the same shape as RobustScaler), fused ahead
of a tree ensemble.  For float32 input each step is computed in double precision and rounded
to float32, the way numpy evaluates float32 data against float64 parameters:
  MINMAX        x1 = f32(x * a);  x' = f32(x1 + b)
  CENTER_SCALE  x1 = f32(x - a);  x' = f32(x1 / b)
  BINARIZE      x' = 1 if x > a else 0     (NaN -> 0)
The forest's thresholds then apply to x'.
"""
from __future__ import annotations

import numpy as np

NONE, MINMAX, CENTER_SCALE, BINARIZE = 0, 1, 2, 3


def apply(kind: int, a, b, X: np.ndarray) -> np.ndarray:
    X = np.asarray(X, np.float32)
    if kind == NONE:
        return X.copy()
    a = np.asarray(a, np.float64)[None, :]
    if kind == MINMAX:
        x1 = (X.astype(np.float64) * a).astype(np.float32)
        return (x1.astype(np.float64) + np.asarray(b, np.float64)[None, :]).astype(np.float32)
    if kind == CENTER_SCALE:
        x1 = (X.astype(np.float64) - a).astype(np.float32)
        return (x1.astype(np.float64) / np.asarray(b, np.float64)[None, :]).astype(np.float32)
    if kind == BINARIZE:
        return (X.astype(np.float64) > a).astype(np.float32)
    raise ValueError(kind)
