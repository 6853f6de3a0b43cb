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
  NORMALIZE     s = sum over f = 0, 1, ..., F-1 of double(x_f)^2, one double add at a time in
                feature order;  n = sqrt(s) (1 when s == 0);  x' = f32(x / n)
NORMALIZE is the Normalizer's unit L2 row norm.  The squares of float32 values are exact in
double and their sum cannot overflow, so x' is within a hair of x / ||x|| rounded once; the
fixed summation order makes the double norm itself reproducible.  A NaN in the row makes the
whole row NaN; an infinity makes its own entry NaN and every finite entry zero.
The forest's thresholds then apply to x'.
"""
from __future__ import annotations

import numpy as np

NONE, MINMAX, CENTER_SCALE, BINARIZE, NORMALIZE = 0, 1, 2, 3, 4


def row_norms(X: np.ndarray) -> np.ndarray:
    """The double L2 norm of each row, summed one feature at a time in feature order (1.0 for
    an all-zero row, which the Normalizer leaves unchanged)."""
    X = np.asarray(X, np.float32)
    s = np.zeros(X.shape[0], np.float64)
    for f in range(X.shape[1]):
        xf = X[:, f].astype(np.float64)
        s = s + xf * xf
    n = np.sqrt(s)
    n[s == 0.0] = 1.0
    return n


def apply(kind: int, a, b, X: np.ndarray) -> np.ndarray:
    X = np.asarray(X, np.float32)
    if kind == NONE:
        return X.copy()
    if kind == NORMALIZE:
        return (X.astype(np.float64) / row_norms(X)[:, None]).astype(np.float32)
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
