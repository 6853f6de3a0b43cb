"""CPU oracle for batched tree-ensemble prediction -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The library (``paper_2405_12491_amd``)
never does; it shares no code with it.

``forest_oracle.c`` holds the arithmetic (see its header for the definition it
follows and the conventions it takes where the paper is silent).  This wrapper
only compiles it with gcc and marshals numpy arrays through ctypes; rows may be
split across threads, each thread evaluating its own rows with identical
per-row arithmetic.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "forest_oracle.c")
_LIB_PATH = os.path.join(_HERE, "_forest_oracle.so")
GCC_FLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared", "-std=c99"]

_lib = None
_lock = threading.Lock()


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle with gcc (no FMA contraction, no fast-math)."""
    tmp = f"{out}.{os.getpid()}.tmp"  # one per process: parallel test workers build at once
    cmd = ["gcc", *GCC_FLAGS, "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def load(path: Optional[str] = None):
    global _lib
    with _lock:
        if path is None and _lib is not None:
            return _lib
        p = path or _LIB_PATH
        if path is None and (not os.path.exists(p) or os.path.getmtime(p) < os.path.getmtime(_SRC)):
            build()
        lib = ctypes.CDLL(p)
        P = ctypes.c_void_p
        lib.oracle_predict.restype = ctypes.c_int
        lib.oracle_predict.argtypes = [ctypes.c_int32, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_int32,
                                       P, ctypes.c_int32, ctypes.c_int32, P, P, ctypes.c_int64, P, P, P]
        if path is None:
            _lib = lib
        return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    pass


def predict(forest, X: np.ndarray, want_leaves: bool = False, threads: int = 1, lib=None):
    """Return (out float64 [n, K], leaves int32 [n, T] or None, visits int).

    ``forest`` is a ``synth.Forest`` (or any object with the same fields)."""
    lib = lib or load()
    X = np.ascontiguousarray(X, dtype=np.float32)
    n = X.shape[0]
    K = int(forest.n_classes)
    T = int(forest.n_trees)
    if X.ndim != 2 or X.shape[1] != forest.n_features:
        raise OracleError("X shape does not match the forest's feature count")
    arrs = dict(
        offs=np.ascontiguousarray(forest.tree_offsets, np.int64),
        feat=np.ascontiguousarray(forest.feature, np.int32),
        thr=np.ascontiguousarray(forest.threshold, np.float32),
        left=np.ascontiguousarray(forest.left, np.int32),
        right=np.ascontiguousarray(forest.right, np.int32),
        val=np.ascontiguousarray(forest.value, np.float32),
        tc=None if forest.tree_class is None else np.ascontiguousarray(forest.tree_class, np.int32),
        base=None if forest.base_score is None else np.ascontiguousarray(forest.base_score, np.float32),
    )
    out = np.empty((n, K), np.float64)
    leaves = np.empty((n, T), np.int32) if want_leaves else None
    threads = max(1, min(int(threads), max(n, 1)))
    bounds = np.linspace(0, n, threads + 1).astype(np.int64)
    visits = [0] * threads
    rcs = [0] * threads

    def work(i):
        a, b = int(bounds[i]), int(bounds[i + 1])
        v = ctypes.c_int64(0)
        rcs[i] = lib.oracle_predict(
            T, _ptr(arrs["offs"]), _ptr(arrs["feat"]), _ptr(arrs["thr"]), _ptr(arrs["left"]),
            _ptr(arrs["right"]), _ptr(arrs["val"]), int(forest.n_features), K, _ptr(arrs["tc"]),
            int(forest.aggregate), int(forest.transform), _ptr(arrs["base"]),
            _ptr(X[a:b]) if b > a else _ptr(X), b - a, _ptr(out[a:b]) if b > a else _ptr(out),
            _ptr(leaves[a:b]) if (leaves is not None and b > a) else None, ctypes.byref(v))
        visits[i] = v.value

    if threads == 1:
        work(0)
    else:
        ts = [threading.Thread(target=work, args=(i,)) for i in range(threads)]
        for t in ts:
            t.start()
        for t in ts:
            t.join()
    for rc in rcs:
        if rc != 0:
            raise OracleError(f"oracle_predict failed with code {rc}")
    return out, leaves, int(sum(visits))
