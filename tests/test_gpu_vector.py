"""GPU parity of vector-leaf forests (tree classifiers): averaged class vectors, labels and leaf
ids on every kernel family that takes them, against the vector oracle."""
import dataclasses

import numpy as np
import pytest

import paper_2405_12491_amd as B
from oracle import sparse as S
from oracle import vector as V
from parity_util import assert_leaves, assert_scores, check_labels, to_dev
from synth import (AGG_SUM, XFORM_SOFTMAX, make_workload, random_tiny_forest,
                   with_vector_leaves)

pytestmark = pytest.mark.gpu

KERNELS = [B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _case(name, rng):
    if name == "tiny_ragged":
        base = random_tiny_forest(rng, 40, 9, max_depth=9)
        X = rng.standard_normal((1300, 9)).astype(np.float32)
        X[5, 3] = np.nan
        return with_vector_leaves(base, 4, rng), X
    # K = 2 and 3: class rows staged with the tree blocks; 5 and 10: rows read from L2
    K, n = {"rf_d8": (5, 1200), "mc_gbdt_d8": (10, 200), "ragged_d12": (3, 200),
            "gbdt_d6": (2, 1500), "rf_d8_k3": (3, 1100)}[name]
    w = make_workload(name.split("_k")[0], n)
    return with_vector_leaves(w.forest, K, rng), w.X()


@pytest.mark.parametrize("name", ["rf_d8", "rf_d8_k3", "mc_gbdt_d8", "ragged_d12", "gbdt_d6",
                                  "tiny_ragged", "tiny_ragged_chunked"])
def test_vector_forest(name, monkeypatch):
    import torch
    if name.endswith("_chunked"):   # ragged trees through LDS chunks instead of global records
        monkeypatch.setenv("BRIDGER_GLOBAL", "0")
        name = name[:-len("_chunked")]
    rng = np.random.default_rng(len(name))
    model, X = _case(name, rng)
    ref, ref_lv = V.predict(model, X, threads=8)
    Xd = to_dev(X)
    with B.Forest(model) as f:
        ran = 0
        for k in KERNELS:
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            what = f"{name} vector {B.KERNEL_NAMES[k]}"
            print(f"[vec] {what}", flush=True)
            out = f.predict(Xd)
            lab = f.predict_labels(Xd)
            lv = f.predict_leaves(Xd)
            torch.cuda.synchronize()
            assert_scores(out.cpu().numpy(), ref, what + " scores")
            check_labels(lab.cpu().numpy(), ref, what + " labels")
            assert_leaves(lv.cpu().numpy(), ref_lv, what + " leaves")
            ran += 1
        assert ran >= 2
        with pytest.raises(B.BridgerError) as e:
            f.kernel = B.BRIDGER_KERNEL_GEMM
        assert e.value.status == B.BRIDGER_ERR_UNSUPPORTED
        # bins and CSR rows reach the same kernels
        f.kernel = B.BRIDGER_KERNEL_AUTO
        if f.bin_info()["bin_bytes"] and f.kernel in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
            out = f.predict_binned(f.bin(Xd))
            torch.cuda.synchronize()
            assert_scores(out.cpu().numpy(), ref, name + " vector binned")
        if f.kernel in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
            nz = np.nonzero(np.where(np.isnan(X), 1.0, X))
            ip = np.concatenate([[0], np.cumsum(np.bincount(nz[0], minlength=X.shape[0]))]).astype(np.int64)
            ix, vv = nz[1].astype(np.int32), X[nz].astype(np.float32)
            assert np.array_equal(np.nan_to_num(S.densify(ip, ix, vv, *X.shape), nan=7.0),
                                  np.nan_to_num(X, nan=7.0))
            d = lambda a: torch.from_numpy(a).cuda()
            out = f.predict_csr(d(ip), d(ix), d(vv), X.shape[0])
            torch.cuda.synchronize()
            assert_scores(out.cpu().numpy(), ref, name + " vector csr")


def test_vector_sum_base_and_softmax():
    import torch
    rng = np.random.default_rng(9)
    base = random_tiny_forest(rng, 25, 7, max_depth=8)
    model = with_vector_leaves(base, 6, rng, aggregate=AGG_SUM, transform=XFORM_SOFTMAX)
    model = dataclasses.replace(model, base_score=rng.standard_normal(6).astype(np.float32))
    X = rng.standard_normal((1000, 7)).astype(np.float32)
    ref, _ = V.predict(model, X)
    Xd = to_dev(X)
    with B.Forest(model) as f:
        for k in KERNELS:
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            out = f.predict(Xd)
            torch.cuda.synchronize()
            assert_scores(out.cpu().numpy(), ref, f"sum+softmax {B.KERNEL_NAMES[k]}")
