"""GPU parity of fused preprocessing: predictions (every kernel family) and bins of
preprocessed rows against the oracle run on the oracle-preprocessed rows."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from oracle import binning
from oracle import preprocess as P
from parity_util import assert_leaves, assert_scores, gpu_predict, oracle_predict, to_dev
from synth import make_workload

pytestmark = pytest.mark.gpu

KERNELS = [B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT,
           B.BRIDGER_KERNEL_GEMM]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _params(kind, X, rng):
    from sklearn.preprocessing import MinMaxScaler, RobustScaler
    Xf = np.nan_to_num(X, nan=0.0, posinf=0.0, neginf=0.0)   # scalers are fitted on finite data
    if kind == P.MINMAX:
        s = MinMaxScaler(feature_range=(-2, 2)).fit(Xf)
        return s.scale_, s.min_
    if kind == P.CENTER_SCALE:
        s = RobustScaler().fit(Xf)
        return s.center_, s.scale_
    if kind == P.NORMALIZE:
        return None, None
    return rng.standard_normal(X.shape[1]) * 0.5, None


@pytest.mark.parametrize("kind", [P.MINMAX, P.CENTER_SCALE, P.BINARIZE, P.NORMALIZE])
@pytest.mark.parametrize("name,n", [("gbdt_d6", 1500), ("rf_d8", 700), ("ragged_d12", 150),
                                    ("mc_gbdt_d8", 150), ("shallow_d3", 1100), ("ragged_rf_28", 700),
                                    ("ragged_rf_28_chunked", 700)])
def test_fused_preprocessing(kind, name, n, monkeypatch):
    import torch
    if name.endswith("_chunked"):   # ragged trees through LDS chunks instead of global records
        monkeypatch.setenv("BRIDGER_GLOBAL", "0")
        name = name[:-len("_chunked")]
    rng = np.random.default_rng(kind * 10 + n)
    w = make_workload(name, n)
    X = w.X()
    X[3, 1] = np.nan
    X[4, 2] = np.inf
    X[5, 0] = -np.inf
    a, b = _params(kind, X, rng)
    Xp = P.apply(kind, a, b, X)
    ref, ref_lv = oracle_predict(w.forest, Xp, leaves=True)
    Xd = to_dev(X)
    with B.Forest(w.forest) as f:
        f.set_preprocess(kind, a, b)
        for k in KERNELS:
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            what = f"{name} pre={kind} {B.KERNEL_NAMES[k]}"
            print(f"[pre] {what}", flush=True)
            assert_scores(gpu_predict(f, Xd), ref, what + " scores")
            assert_leaves(gpu_predict(f, Xd, leaves=True), ref_lv, what + " leaves")
        # bins of the preprocessed rows, and prediction on them
        f.kernel = B.BRIDGER_KERNEL_AUTO
        if f.bin_info()["bin_bytes"] and f.kernel in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
            q = f.bin(Xd)
            out = f.predict_binned(q)
            torch.cuda.synchronize()
            bb = f.bin_info()["bin_bytes"]
            got = q.cpu().numpy().view(np.uint8 if bb == 1 else np.uint16).astype(np.int64)
            assert np.array_equal(got, binning.bin_rows(binning.tables(w.forest), Xp)), name + " bins"
            assert_scores(out.cpu().numpy().astype(np.float64), ref, f"{name} pre={kind} binned")
        # switching the preprocessing off restores the plain prediction
        f.set_preprocess(B.BRIDGER_PRE_NONE)
        ref0, _ = oracle_predict(w.forest, X)
        assert_scores(gpu_predict(f, Xd), ref0, f"{name} preprocessing off")


@pytest.mark.parametrize("name,n", [("gbdt_d6", 1500), ("rf_d8", 700), ("ragged_d12", 150),
                                    ("mc_gbdt_d8", 150)])
def test_normalize_at_ties(name, n):
    """Normalizer with every threshold equal to some row's normalized feature value, so a last-bit
    difference anywhere in the norm or the divide changes a leaf."""
    import dataclasses
    import torch
    rng = np.random.default_rng(n + 7)
    w = make_workload(name, n)
    X = w.X()
    X[2] = 0.0                                  # zero row: left unchanged
    Xp = P.apply(P.NORMALIZE, None, None, X)
    m = w.forest
    thr = m.threshold.copy()
    rows = rng.integers(0, n, thr.shape[0])
    thr[:] = Xp[rows, np.clip(m.feature, 0, X.shape[1] - 1)]
    model = dataclasses.replace(m, threshold=thr)
    ref, ref_lv = oracle_predict(model, Xp, leaves=True)
    Xd = to_dev(X)
    with B.Forest(model) as f:
        f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)
        for k in KERNELS:
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            what = f"{name} normalize ties {B.KERNEL_NAMES[k]}"
            print(f"[pre] {what}", flush=True)
            assert_scores(gpu_predict(f, Xd), ref, what + " scores")
            assert_leaves(gpu_predict(f, Xd, leaves=True), ref_lv, what + " leaves")
        f.kernel = B.BRIDGER_KERNEL_AUTO
        if f.bin_info()["bin_bytes"]:
            q = f.bin(Xd)
            torch.cuda.synchronize()
            bb = f.bin_info()["bin_bytes"]
            got = q.cpu().numpy().view(np.uint8 if bb == 1 else np.uint16).astype(np.int64)
            assert np.array_equal(got, binning.bin_rows(binning.tables(model), Xp)), name + " bins"


def test_normalize_concurrent_streams():
    """The Normalizer's row norms live in stream-ordered scratch taken per call: predictions in
    flight on two streams at once (and many calls in a row) each get their own norms."""
    import torch
    rng = np.random.default_rng(5)
    w = make_workload("gbdt_d6", 20_000)
    X1 = w.X()
    X2 = (rng.standard_normal(X1.shape) * 3).astype(np.float32)
    ref1, _ = oracle_predict(w.forest, P.apply(P.NORMALIZE, None, None, X1))
    ref2, _ = oracle_predict(w.forest, P.apply(P.NORMALIZE, None, None, X2))
    d1, d2 = to_dev(X1), to_dev(X2)
    with B.Forest(w.forest) as f:
        f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        outs1, outs2 = [], []
        for _ in range(8):
            with torch.cuda.stream(s1):
                outs1.append(f.predict(d1))
            with torch.cuda.stream(s2):
                outs2.append(f.predict(d2))
        torch.cuda.synchronize()
        for o in outs1:
            assert_scores(o.cpu().numpy(), ref1, "stream 1")
        for o in outs2:
            assert_scores(o.cpu().numpy(), ref2, "stream 2")
