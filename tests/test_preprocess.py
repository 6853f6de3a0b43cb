"""Fused preprocessing on the CPU: the preprocessing oracle against scikit-learn's scalers
(bit for bit on float32 data), planted mistakes, and the ABI's argument checks."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from oracle import preprocess as P
from synth import make_workload


def _data(seed=0, n=4000, F=6):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((n, F)) * rng.uniform(0.01, 1000, F)).astype(np.float32)
    X[rng.random(X.shape) < 0.01] = 0.0
    X[rng.random(X.shape) < 0.01] = -0.0
    return X


def _sklearn_cases(X):
    from sklearn.preprocessing import Binarizer, MinMaxScaler, RobustScaler, StandardScaler
    mm = MinMaxScaler().fit(X)
    st = StandardScaler().fit(X)
    rb = RobustScaler().fit(X)
    t = float(np.float32(0.25))
    return [
        ("MinMaxScaler", P.MINMAX, mm.scale_, mm.min_, mm.transform(X)),
        ("StandardScaler", P.CENTER_SCALE, st.mean_, st.scale_, st.transform(X)),
        ("RobustScaler", P.CENTER_SCALE, rb.center_, rb.scale_, rb.transform(X)),
        ("Binarizer", P.BINARIZE, np.full(X.shape[1], t), None, Binarizer(threshold=t).transform(X)),
    ]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_oracle_matches_sklearn_bit_for_bit(seed):
    X = _data(seed)
    for name, kind, a, b, ref in _sklearn_cases(X):
        got = P.apply(kind, a, b, X)
        assert ref.dtype == np.float32, name
        assert np.array_equal(got.view(np.uint32), ref.astype(np.float32).view(np.uint32)), name


def test_pins_reject_plausible_mistakes():
    X = _data(7, n=20000)
    cases = {c[0]: c for c in _sklearn_cases(X)}

    def one_rounding_minmax(a, b, X):     # no rounding between the multiply and the add
        return (X.astype(np.float64) * a + b).astype(np.float32)

    def divide_then_subtract(a, b, X):    # x/b - a/b
        return (X.astype(np.float64) / b - a / b).astype(np.float32)

    def float32_params(a, b, X):          # parameters rounded to float32 first
        return P.apply(P.CENTER_SCALE, np.float32(a), np.float32(b), X)

    def ge_binarize(a, b, X):             # >= instead of >
        return (X.astype(np.float64) >= a).astype(np.float32)

    for name, fn in (("MinMaxScaler", one_rounding_minmax), ("StandardScaler", divide_then_subtract),
                     ("StandardScaler", float32_params)):
        _, _, a, b, ref = cases[name]
        assert not np.array_equal(fn(np.asarray(a, np.float64)[None, :], np.asarray(b, np.float64)[None, :], X)
                                  .view(np.uint32), ref.astype(np.float32).view(np.uint32)), name
    Xt = X.copy()
    Xt[:100, :] = np.float32(0.25)          # ties with the threshold
    _, _, a, _, _ = cases["Binarizer"]
    from sklearn.preprocessing import Binarizer
    ref = Binarizer(threshold=float(a[0])).transform(Xt)
    assert not np.array_equal(ge_binarize(np.asarray(a)[None, :], None, Xt), ref)
    assert np.array_equal(P.apply(P.BINARIZE, a, None, Xt), ref)


def test_set_preprocess_argument_errors():
    w = make_workload("gbdt_d6", 10)
    with B.Forest(w.forest, host_only=True) as f:
        a = np.zeros(28)
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_set_preprocess(f.handle, 9, a, a)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_set_preprocess(f.handle, B.BRIDGER_PRE_MINMAX, a, None)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_set_preprocess(f.handle, B.BRIDGER_PRE_BINARIZE, None, None)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        f.set_preprocess(B.BRIDGER_PRE_BINARIZE, a)
        f.set_preprocess(B.BRIDGER_PRE_NONE)
