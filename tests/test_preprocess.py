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


def _exact_normalized(X):
    """x / ||x|| in exact decimal arithmetic (80 digits) for each element."""
    from decimal import Decimal, getcontext
    getcontext().prec = 80
    out = []
    for row in X.astype(np.float64):
        s = sum(Decimal(float(v)) * Decimal(float(v)) for v in row)
        n = s.sqrt() if s != 0 else Decimal(1)
        out.append([Decimal(float(v)) / n for v in row])
    return out


def _within_half_ulp(got, exact):
    """True where the float32 `got` is within half an ulp (plus 2^-25 of it) of the exact value,
    i.e. the correctly rounded result unless the value sits on a rounding midpoint."""
    from decimal import Decimal
    ok = np.zeros(got.shape, bool)
    for i, row in enumerate(exact):
        for j, q in enumerate(row):
            g = np.float32(got[i, j])
            half = Decimal(float(np.spacing(np.abs(g)))) / 2
            ok[i, j] = abs(Decimal(float(g)) - q) <= half * (1 + Decimal(2) ** -25)
    return ok


def test_normalize_is_the_correctly_rounded_unit_row():
    X = _data(3, n=300)
    got = P.apply(P.NORMALIZE, None, None, X)
    assert got.dtype == np.float32
    assert _within_half_ulp(got, _exact_normalized(X)).all()


def test_normalize_pins_reject_plausible_mistakes():
    X = _data(4, n=300)
    exact = _exact_normalized(X)

    def f32_sum(X):                       # norm accumulated in float32
        s = np.zeros(X.shape[0], np.float32)
        for f in range(X.shape[1]):
            s = s + X[:, f] * X[:, f]
        return (X.astype(np.float64) / np.sqrt(s.astype(np.float64))[:, None]).astype(np.float32)

    def f32_norm(X):                      # double norm rounded to float32 before the divide
        return (X.astype(np.float64) / P.row_norms(X).astype(np.float32)[:, None]).astype(np.float32)

    def dropped_term(X):                  # last feature left out of the norm
        n = P.row_norms(X[:, :-1])
        return (X.astype(np.float64) / n[:, None]).astype(np.float32)

    def f32_divide(X):                    # the divide done in float32
        return (X / P.row_norms(X).astype(np.float32)[:, None]).astype(np.float32)

    def l1(X):                            # wrong norm
        n = np.abs(X.astype(np.float64)).sum(1)
        return (X.astype(np.float64) / n[:, None]).astype(np.float32)

    for fn in (f32_sum, f32_norm, f32_divide, dropped_term, l1):
        assert not _within_half_ulp(fn(X), exact).all(), fn.__name__


def test_normalize_against_sklearn_and_special_rows():
    from sklearn.preprocessing import Normalizer
    X = _data(5, n=4000)
    X[7] = 0.0
    X[8] = -0.0
    got = P.apply(P.NORMALIZE, None, None, X)
    ref = Normalizer().fit(X).transform(X).astype(np.float32)
    # scikit-learn computes the norm in float32: a few ulps apart at most, mostly equal
    d = np.abs(got.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
    assert d.max() <= 4 and (d == 0).mean() > 0.5
    assert np.array_equal(got[7:9].view(np.uint32), X[7:9].view(np.uint32))   # zero rows kept
    S = np.array([[3, 4, 0, 0], [0, -5, 0, 0], [1, 1, 1, 1], [np.nan, 1, 2, 3],
                  [np.inf, 1, -2, 0], [3e38, 3e38, 0, 0], [1e-45, 0, 0, 0]], np.float32)
    g = P.apply(P.NORMALIZE, None, None, S)
    f = np.float32
    assert g[0].tolist() == [f(0.6), f(0.8), 0.0, 0.0]
    assert g[1].tolist() == [0.0, -1.0, 0.0, 0.0]
    assert g[2].tolist() == [0.5] * 4
    assert np.isnan(g[3]).all()
    assert np.isnan(g[4, 0]) and g[4, 1:].tolist() == [0.0, -0.0, 0.0]
    assert g[5].tolist() == [f(np.sqrt(0.5)), f(np.sqrt(0.5)), 0.0, 0.0]    # no overflow
    assert g[6].tolist() == [1.0, 0.0, 0.0, 0.0]                            # no underflow


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
        f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)          # no parameters
        f.set_preprocess(B.BRIDGER_PRE_NONE)
