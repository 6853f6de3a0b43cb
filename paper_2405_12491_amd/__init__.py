"""MI355X tree-ensemble prediction: Python binding of the C ABI in include/bridger.h.

The functions named ``bridger_*`` marshal arguments to the entry points of the same
name in ``libbridger.so`` (built by ``paper_2405_12491_amd.build``); every step of
prediction runs in the library's HIP kernels.  ``Forest`` is a small convenience
wrapper that takes numpy arrays for the model and torch CUDA tensors for the rows,
using torch only for device memory and the current stream.  There is no CPU
fallback: if the library is missing, importing the binding's functions raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbridger.so")

BRIDGER_OK = 0
BRIDGER_ERR_INVALID_ARGUMENT = 1
BRIDGER_ERR_INVALID_FOREST = 2
BRIDGER_ERR_UNSUPPORTED = 3
BRIDGER_ERR_OUT_OF_MEMORY = 4
BRIDGER_ERR_DEVICE = 5
STATUS_NAMES = {0: "OK", 1: "INVALID_ARGUMENT", 2: "INVALID_FOREST", 3: "UNSUPPORTED",
                4: "OUT_OF_MEMORY", 5: "DEVICE"}

BRIDGER_AGG_SUM, BRIDGER_AGG_MEAN = 0, 1
BRIDGER_XFORM_IDENTITY, BRIDGER_XFORM_SIGMOID, BRIDGER_XFORM_SOFTMAX = 0, 1, 2
BRIDGER_KERNEL_AUTO, BRIDGER_KERNEL_PERFECT, BRIDGER_KERNEL_RAGGED, BRIDGER_KERNEL_DIRECT = 0, 1, 2, 3
BRIDGER_KERNEL_GEMM = 4
KERNEL_NAMES = {0: "auto", 1: "perfect", 2: "ragged", 3: "direct", 4: "gemm"}
BRIDGER_CREATE_HOST_ONLY = 1
BRIDGER_CREATE_VECTOR_LEAVES = 2
BRIDGER_PRE_NONE, BRIDGER_PRE_MINMAX, BRIDGER_PRE_CENTER_SCALE, BRIDGER_PRE_BINARIZE = 0, 1, 2, 3
BRIDGER_PRE_NORMALIZE = 4

_lib = None


def _launch_stream(device) -> int:
    """Raw handle of torch's current stream on ``device`` (where the kernels are launched).
    torch's raw-stream query costs about 0.1 us against about 2 us for the stream object, which
    matters for small batches; the public query serves if the raw one is absent."""
    import torch
    try:
        return torch._C._cuda_getCurrentRawStream(device.index)
    except AttributeError:
        return torch.cuda.current_stream(device).cuda_stream


class BridgerError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def load_library(path: Optional[str] = None):
    """Load libbridger.so (raises OSError if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise OSError(f"{p} not found: build it with `python -m paper_2405_12491_amd.build`")
    lib = ctypes.CDLL(p)
    P, I32, I64, U32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    create_args = [I32, P, P, P, P, P, P, I32, I32, P, I32, I32, P]
    lib.bridger_forest_create.argtypes = create_args + [P]
    lib.bridger_forest_create_ex.argtypes = create_args + [U32, P]
    lib.bridger_forest_predict.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_predict_leaves.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_predict_noalloc.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_info.argtypes = [P, P, P, P, P, P]
    lib.bridger_forest_bin_info.argtypes = [P, P, P]
    lib.bridger_forest_predict_labels.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_predict_csr.argtypes = [P, P, P, P, I64, I32, P, P]
    lib.bridger_forest_predict_csr_leaves.argtypes = [P, P, P, P, I64, I32, P, P]
    lib.bridger_forest_set_preprocess.argtypes = [P, I32, P, P]
    lib.bridger_forest_bin.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_predict_binned.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_predict_binned_leaves.argtypes = [P, P, I64, I32, P, P]
    lib.bridger_forest_set_kernel.argtypes = [P, I32]
    lib.bridger_forest_get_kernel.argtypes = [P, P]
    lib.bridger_forest_plan.argtypes = [P, I64, P, P, P, P, P, P, P, P]
    lib.bridger_forest_packed.argtypes = [P, I32, P, P]
    lib.bridger_forest_destroy.argtypes = [P]
    lib.bridger_forest_destroy.restype = None
    lib.bridger_last_error.argtypes = []
    lib.bridger_last_error.restype = ctypes.c_char_p
    for name in ("bridger_forest_create", "bridger_forest_create_ex", "bridger_forest_predict",
                 "bridger_forest_predict_leaves", "bridger_forest_info", "bridger_forest_set_kernel",
                 "bridger_forest_get_kernel", "bridger_forest_plan", "bridger_forest_packed",
                 "bridger_forest_bin_info", "bridger_forest_bin", "bridger_forest_predict_binned",
                 "bridger_forest_predict_binned_leaves", "bridger_forest_set_preprocess",
                 "bridger_forest_predict_labels", "bridger_forest_predict_csr",
                 "bridger_forest_predict_csr_leaves"):
        getattr(lib, name).restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def _check(status: int, where: str):
    if status != BRIDGER_OK:
        msg = load_library().bridger_last_error().decode(errors="replace")
        raise BridgerError(status, where, msg)


def _vp(a):
    if a is None:
        return None
    if isinstance(a, int):
        return ctypes.c_void_p(a)
    return a.ctypes.data_as(ctypes.c_void_p)


# ------------------------------------------------------------- raw entry points
def bridger_forest_create(n_trees, tree_offsets, feature, threshold, left, right, value,
                          n_features, n_classes, tree_class, aggregate, transform, base_score,
                          flags: int = 0) -> ctypes.c_void_p:
    """Returns the opaque handle; arrays are numpy arrays of the documented dtypes.  A 2-D
    ``value`` [N, n_classes] makes a vector-leaf forest (BRIDGER_CREATE_VECTOR_LEAVES)."""
    lib = load_library()
    h = ctypes.c_void_p()
    if np.ndim(value) == 2:
        flags |= BRIDGER_CREATE_VECTOR_LEAVES
    arrs = [np.ascontiguousarray(tree_offsets, np.int64), np.ascontiguousarray(feature, np.int32),
            np.ascontiguousarray(threshold, np.float32), np.ascontiguousarray(left, np.int32),
            np.ascontiguousarray(right, np.int32), np.ascontiguousarray(value, np.float32)]
    tc = None if tree_class is None else np.ascontiguousarray(tree_class, np.int32)
    bs = None if base_score is None else np.ascontiguousarray(base_score, np.float32)
    st = lib.bridger_forest_create_ex(int(n_trees), *[_vp(a) for a in arrs], int(n_features),
                                      int(n_classes), _vp(tc), int(aggregate), int(transform),
                                      _vp(bs), int(flags), ctypes.byref(h))
    _check(st, "bridger_forest_create")
    return h


def bridger_forest_predict(h, X_ptr: int, n_rows: int, n_features: int, out_ptr: int, stream: int = 0):
    _check(load_library().bridger_forest_predict(h, ctypes.c_void_p(X_ptr), int(n_rows),
                                                 int(n_features), ctypes.c_void_p(out_ptr),
                                                 ctypes.c_void_p(stream)), "bridger_forest_predict")


NOALLOC_MAX_ROWS = 2097152   # BRIDGER_NOALLOC_MAX_ROWS


def bridger_forest_predict_noalloc(h, X_ptr: int, n_rows: int, n_features: int, out_ptr: int,
                                   stream: int = 0):
    """The allocation-free predict (at most NOALLOC_MAX_ROWS rows per call)."""
    _check(load_library().bridger_forest_predict_noalloc(h, ctypes.c_void_p(X_ptr), int(n_rows),
                                                         int(n_features), ctypes.c_void_p(out_ptr),
                                                         ctypes.c_void_p(stream)),
           "bridger_forest_predict_noalloc")


def bridger_forest_predict_leaves(h, X_ptr: int, n_rows: int, n_features: int, out_ptr: int,
                                  stream: int = 0):
    _check(load_library().bridger_forest_predict_leaves(h, ctypes.c_void_p(X_ptr), int(n_rows),
                                                        int(n_features), ctypes.c_void_p(out_ptr),
                                                        ctypes.c_void_p(stream)),
           "bridger_forest_predict_leaves")


def bridger_forest_set_preprocess(h, kind: int, a=None, b=None):
    """a, b: per-feature parameters (float64 numpy arrays) or None."""
    av = None if a is None else np.ascontiguousarray(a, np.float64)
    bv = None if b is None else np.ascontiguousarray(b, np.float64)
    _check(load_library().bridger_forest_set_preprocess(h, int(kind), _vp(av), _vp(bv)),
           "bridger_forest_set_preprocess")


def bridger_forest_bin_info(h) -> dict:
    b, n = ctypes.c_int32(), ctypes.c_int64()
    _check(load_library().bridger_forest_bin_info(h, ctypes.byref(b), ctypes.byref(n)),
           "bridger_forest_bin_info")
    return {"bin_bytes": b.value, "n_thresholds": n.value}


def bridger_forest_bin(h, X_ptr: int, n_rows: int, n_features: int, xq_ptr: int, stream: int = 0):
    _check(load_library().bridger_forest_bin(h, ctypes.c_void_p(X_ptr), int(n_rows), int(n_features),
                                             ctypes.c_void_p(xq_ptr), ctypes.c_void_p(stream)),
           "bridger_forest_bin")


def bridger_forest_predict_binned(h, xq_ptr: int, n_rows: int, n_features: int, out_ptr: int,
                                  stream: int = 0):
    _check(load_library().bridger_forest_predict_binned(h, ctypes.c_void_p(xq_ptr), int(n_rows),
                                                        int(n_features), ctypes.c_void_p(out_ptr),
                                                        ctypes.c_void_p(stream)),
           "bridger_forest_predict_binned")


def bridger_forest_predict_binned_leaves(h, xq_ptr: int, n_rows: int, n_features: int,
                                         out_ptr: int, stream: int = 0):
    _check(load_library().bridger_forest_predict_binned_leaves(
        h, ctypes.c_void_p(xq_ptr), int(n_rows), int(n_features), ctypes.c_void_p(out_ptr),
        ctypes.c_void_p(stream)), "bridger_forest_predict_binned_leaves")


def bridger_forest_predict_labels(h, X_ptr: int, n_rows: int, n_features: int, out_ptr: int,
                                  stream: int = 0):
    _check(load_library().bridger_forest_predict_labels(h, ctypes.c_void_p(X_ptr), int(n_rows),
                                                        int(n_features), ctypes.c_void_p(out_ptr),
                                                        ctypes.c_void_p(stream)),
           "bridger_forest_predict_labels")


def bridger_forest_predict_csr(h, indptr_ptr: int, indices_ptr: int, values_ptr: int, n_rows: int,
                               n_features: int, out_ptr: int, stream: int = 0, leaves: bool = False):
    lib = load_library()
    fn = lib.bridger_forest_predict_csr_leaves if leaves else lib.bridger_forest_predict_csr
    _check(fn(h, ctypes.c_void_p(indptr_ptr), ctypes.c_void_p(indices_ptr), ctypes.c_void_p(values_ptr),
              int(n_rows), int(n_features), ctypes.c_void_p(out_ptr), ctypes.c_void_p(stream)),
           "bridger_forest_predict_csr" + ("_leaves" if leaves else ""))


def bridger_forest_info(h) -> dict:
    v = [ctypes.c_int32() for _ in range(5)]
    _check(load_library().bridger_forest_info(h, *[ctypes.byref(x) for x in v]), "bridger_forest_info")
    return dict(zip(("n_trees", "n_features", "n_outputs", "max_depth", "all_perfect"),
                    (x.value for x in v)))


def bridger_forest_set_kernel(h, kernel: int):
    _check(load_library().bridger_forest_set_kernel(h, int(kernel)), "bridger_forest_set_kernel")


def bridger_forest_get_kernel(h) -> int:
    k = ctypes.c_int32()
    _check(load_library().bridger_forest_get_kernel(h, ctypes.byref(k)), "bridger_forest_get_kernel")
    return k.value


def bridger_forest_plan(h, n_rows: int) -> dict:
    i = [ctypes.c_int32() for _ in range(5)]
    d = [ctypes.c_double() for _ in range(3)]
    _check(load_library().bridger_forest_plan(h, int(n_rows), *[ctypes.byref(x) for x in i + d]),
           "bridger_forest_plan")
    keys = ("rows_per_wg", "chunk_bytes", "trees_per_chunk", "n_chunks", "lds_bytes",
            "hbm_bytes", "stage_bytes", "lds_read_bytes")
    return dict(zip(keys, [x.value for x in i + d]))


def bridger_forest_packed(h, which: int, dtype) -> np.ndarray:
    p = ctypes.c_void_p()
    n = ctypes.c_int64()
    _check(load_library().bridger_forest_packed(h, int(which), ctypes.byref(p), ctypes.byref(n)),
           "bridger_forest_packed")
    if n.value == 0:
        return np.zeros(0, dtype)
    buf = (ctypes.c_uint8 * n.value).from_address(p.value)
    return np.frombuffer(bytes(buf), dtype=dtype).copy()


def bridger_forest_destroy(h):
    if h:
        load_library().bridger_forest_destroy(h)


def bridger_last_error() -> str:
    return load_library().bridger_last_error().decode(errors="replace")


# ---------------------------------------------------------------- convenience
class Forest:
    """Owns a forest handle.  ``model`` is any object with the fields of ``synth.Forest``."""

    def __init__(self, model, kernel: int = BRIDGER_KERNEL_AUTO, host_only: bool = False):
        self.n_features = int(model.n_features)
        self.n_classes = int(model.n_classes)
        self.n_trees = int(model.tree_offsets.shape[0] - 1)
        self._h = bridger_forest_create(
            self.n_trees, model.tree_offsets, model.feature, model.threshold, model.left, model.right,
            model.value, self.n_features, self.n_classes, model.tree_class, model.aggregate,
            model.transform, model.base_score, BRIDGER_CREATE_HOST_ONLY if host_only else 0)
        if kernel != BRIDGER_KERNEL_AUTO:
            bridger_forest_set_kernel(self._h, kernel)

    @property
    def handle(self):
        return self._h

    @property
    def kernel(self) -> int:
        return bridger_forest_get_kernel(self._h)

    @kernel.setter
    def kernel(self, k: int):
        bridger_forest_set_kernel(self._h, k)

    def info(self) -> dict:
        return bridger_forest_info(self._h)

    def plan(self, n_rows: int) -> dict:
        return bridger_forest_plan(self._h, n_rows)

    def _check_x(self, X):
        import torch
        if not (isinstance(X, torch.Tensor) and X.is_cuda and X.dtype == torch.float32):
            raise TypeError("X must be a float32 CUDA tensor")
        if X.dim() != 2 or X.shape[1] != self.n_features or not X.is_contiguous():
            raise ValueError("X must be contiguous [n_rows, n_features]")

    def predict(self, X, out=None):
        import torch
        self._check_x(X)
        if out is None:
            out = torch.empty((X.shape[0], self.n_classes), dtype=torch.float32, device=X.device)
        stream = _launch_stream(X.device)
        bridger_forest_predict(self._h, X.data_ptr(), X.shape[0], self.n_features, out.data_ptr(),
                               stream)
        return out

    def predict_csr(self, indptr, indices, values, n_rows: int, out=None, leaves: bool = False):
        """Rows in CSR form: CUDA tensors indptr int64 [n+1], indices int32, values float32."""
        import torch
        for t, dt in ((indptr, torch.int64), (indices, torch.int32), (values, torch.float32)):
            if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dt and t.is_contiguous()):
                raise TypeError("CSR arrays must be contiguous CUDA tensors (int64, int32, float32)")
        if out is None:
            cols = self.n_trees if leaves else self.n_classes
            out = torch.empty((n_rows, cols), dtype=torch.int32 if leaves else torch.float32,
                              device=values.device)
        stream = _launch_stream(values.device)
        bridger_forest_predict_csr(self._h, indptr.data_ptr(), indices.data_ptr(), values.data_ptr(),
                                   n_rows, self.n_features, out.data_ptr(), stream, leaves)
        return out

    def predict_labels(self, X, out=None):
        import torch
        self._check_x(X)
        if out is None:
            out = torch.empty((X.shape[0],), dtype=torch.int32, device=X.device)
        stream = _launch_stream(X.device)
        bridger_forest_predict_labels(self._h, X.data_ptr(), X.shape[0], self.n_features,
                                      out.data_ptr(), stream)
        return out

    def predict_leaves(self, X, out=None):
        import torch
        self._check_x(X)
        if out is None:
            out = torch.empty((X.shape[0], self.n_trees), dtype=torch.int32, device=X.device)
        stream = _launch_stream(X.device)
        bridger_forest_predict_leaves(self._h, X.data_ptr(), X.shape[0], self.n_features,
                                      out.data_ptr(), stream)
        return out

    def set_preprocess(self, kind: int, a=None, b=None):
        for v in (a, b):
            if v is not None and len(v) != self.n_features:
                raise ValueError("preprocessing parameters need one value per feature")
        bridger_forest_set_preprocess(self._h, kind, a, b)

    def bin_info(self) -> dict:
        return bridger_forest_bin_info(self._h)

    def bin(self, X, out=None):
        """Bins of X (uint8 or uint16 CUDA tensor [n, F]) for predict_binned."""
        import torch
        self._check_x(X)
        bb = self.bin_info()["bin_bytes"]
        if bb == 0:
            raise BridgerError(BRIDGER_ERR_UNSUPPORTED, "Forest.bin", "forest cannot be binned")
        if out is None:
            out = torch.empty((X.shape[0], self.n_features),
                              dtype=torch.uint8 if bb == 1 else torch.int16, device=X.device)
        stream = _launch_stream(X.device)
        bridger_forest_bin(self._h, X.data_ptr(), X.shape[0], self.n_features, out.data_ptr(), stream)
        return out

    def _check_q(self, Xq):
        import torch
        if not (isinstance(Xq, torch.Tensor) and Xq.is_cuda and Xq.element_size() in (1, 2)):
            raise TypeError("Xq must be a CUDA tensor of 8- or 16-bit bins")
        if Xq.dim() != 2 or Xq.shape[1] != self.n_features or not Xq.is_contiguous():
            raise ValueError("Xq must be contiguous [n_rows, n_features]")
        if Xq.element_size() != self.bin_info()["bin_bytes"]:
            raise ValueError("Xq element size differs from the forest's bin size")

    def predict_binned(self, Xq, out=None):
        import torch
        self._check_q(Xq)
        if out is None:
            out = torch.empty((Xq.shape[0], self.n_classes), dtype=torch.float32, device=Xq.device)
        stream = _launch_stream(Xq.device)
        bridger_forest_predict_binned(self._h, Xq.data_ptr(), Xq.shape[0], self.n_features,
                                      out.data_ptr(), stream)
        return out

    def predict_binned_leaves(self, Xq, out=None):
        import torch
        self._check_q(Xq)
        if out is None:
            out = torch.empty((Xq.shape[0], self.n_trees), dtype=torch.int32, device=Xq.device)
        stream = _launch_stream(Xq.device)
        bridger_forest_predict_binned_leaves(self._h, Xq.data_ptr(), Xq.shape[0], self.n_features,
                                             out.data_ptr(), stream)
        return out

    def close(self):
        if self._h:
            bridger_forest_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
