"""The allocation-free predict against bridger_forest_predict, through the C ABI.

Two calls in a row, the second with fewer rows than the first, with the Normalizer fused
(the only prediction whose kernels use scratch: its row norms) and without it; every output
must equal the existing entry point's bit for bit (same kernels, same arithmetic) and lie
within 1e-6 + 1e-5 |oracle| of the oracle.  The device's default stream-ordered memory pool,
which the existing entry point draws its row-norm scratch from, must show no use during the
allocation-free calls.
"""
import ctypes

import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import assert_scores, oracle_predict, to_dev
from synth import make_workload

pytestmark = pytest.mark.gpu

POOL_USED_MEM_HIGH = 8   # hipMemPoolAttrUsedMemHigh


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _hip():
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipDeviceGetDefaultMemPool.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]
    hip.hipMemPoolGetAttribute.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    hip.hipMemPoolSetAttribute.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    return hip


def _pool_high(hip, pool, reset=False):
    v = ctypes.c_uint64(0)
    if reset:
        assert hip.hipMemPoolSetAttribute(pool, POOL_USED_MEM_HIGH, ctypes.byref(v)) == 0
    assert hip.hipMemPoolGetAttribute(pool, POOL_USED_MEM_HIGH, ctypes.byref(v)) == 0
    return v.value


@pytest.mark.parametrize("normalize", [True, False])
def test_noalloc_matches_predict(normalize):
    import torch
    from oracle import preprocess as P
    w = make_workload("gbdt_d6", 9000)
    X = w.X()
    X[3] = 0.0                                  # an all-zero row keeps norm 1
    Xd = to_dev(X)
    hip = _hip()
    pool = ctypes.c_void_p()
    assert hip.hipDeviceGetDefaultMemPool(ctypes.byref(pool), torch.cuda.current_device()) == 0
    stream = torch.cuda.current_stream().cuda_stream
    with B.Forest(w.forest) as f:
        if normalize:
            f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)
        for n in (9000, 2000 + 13):             # the second call is smaller than the first
            print(f"[noalloc] normalize={normalize} rows={n}", flush=True)
            ref_out = torch.full((n, 1), -7.0, dtype=torch.float32, device="cuda")
            got = torch.full((n, 1), -9.0, dtype=torch.float32, device="cuda")
            torch.cuda.synchronize()
            _pool_high(hip, pool, reset=True)
            B.bridger_forest_predict_noalloc(f.handle, Xd.data_ptr(), n, w.n_features,
                                             got.data_ptr(), stream)
            torch.cuda.synchronize()
            assert _pool_high(hip, pool) == 0, "the allocation-free call used the memory pool"
            B.bridger_forest_predict(f.handle, Xd.data_ptr(), n, w.n_features,
                                     ref_out.data_ptr(), stream)
            torch.cuda.synchronize()
            if normalize:   # the existing entry point draws its row norms from the pool
                assert _pool_high(hip, pool) >= 8 * n
            g, r = got.cpu().numpy(), ref_out.cpu().numpy()
            assert np.array_equal(g, r), "allocation-free output differs from predict's"
            Xo = P.apply(B.BRIDGER_PRE_NORMALIZE, None, None, X[:n]) if normalize else X[:n]
            ref, _ = oracle_predict(w.forest, Xo)
            assert_scores(g, ref, f"noalloc normalize={normalize} rows={n}")
