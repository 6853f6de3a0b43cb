"""Vector-leaf forests (tree classifiers) on the CPU: the vector oracle pinned against the
scalar C oracle class by class, against scikit-learn's forest classifiers, and on a
hand-worked stump."""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import vector as V
from synth import AGG_MEAN, AGG_SUM, XFORM_SOFTMAX, make_workload, random_tiny_forest, with_vector_leaves


def _class_slice(f, k):
    """Forest k of the per-class decomposition: the same trees with class k's leaf values."""
    return dataclasses.replace(f, value=np.ascontiguousarray(f.value[:, k]), n_classes=1,
                               tree_class=None, transform=0,
                               base_score=None if f.base_score is None else f.base_score[k:k + 1])


@pytest.mark.parametrize("agg", [AGG_SUM, AGG_MEAN])
def test_each_class_is_the_scalar_forest_of_its_leaf_values(agg):
    rng = np.random.default_rng(11)
    base = random_tiny_forest(rng, 30, 6, max_depth=7)
    f = with_vector_leaves(base, 4, rng, aggregate=agg)
    f = dataclasses.replace(f, base_score=rng.standard_normal(4).astype(np.float32))
    X = rng.standard_normal((500, 6)).astype(np.float32)
    X[3, 2] = np.nan
    out, lv = V.predict(f, X)
    for k in range(4):
        ref, ref_lv, _ = oracle.predict(_class_slice(f, k), X, want_leaves=True)
        assert np.array_equal(out[:, k], ref[:, 0]), k          # same double, bit for bit
        assert np.array_equal(lv, ref_lv)


def test_hand_worked_stump():
    # one stump on feature 0 at 0.5: leaf 1 = (0.25, 0.75), leaf 2 = (1, 0); and a constant tree
    # whose single leaf is (0.5, 0.5); mean of the two trees
    from synth import Forest
    f = Forest(n_features=1, n_classes=2, tree_offsets=np.array([0, 3, 4], np.int64),
               feature=np.array([0, -1, -1, -1], np.int32),
               threshold=np.array([0.5, 0, 0, 0], np.float32),
               left=np.array([1, -1, -1, -1], np.int32), right=np.array([2, -1, -1, -1], np.int32),
               value=np.array([[0, 0], [0.25, 0.75], [1, 0], [0.5, 0.5]], np.float32),
               aggregate=AGG_MEAN)
    X = np.array([[0.5], [0.75], [np.nan], [-np.inf]], np.float32)
    out, lv = V.predict(f, X)
    assert lv.tolist() == [[1, 0], [2, 0], [2, 0], [1, 0]]
    assert out.tolist() == [[0.375, 0.625], [0.75, 0.25], [0.75, 0.25], [0.375, 0.625]]
    assert V.labels(out).tolist() == [1, 0, 0, 1]
    sm, _ = V.predict(dataclasses.replace(f, transform=XFORM_SOFTMAX), X[:1])
    e = np.exp(0.375 - 0.625)
    assert np.allclose(sm[0], [e / (1 + e), 1 / (1 + e)], rtol=1e-15, atol=0)


def _from_sklearn(est, n_features):
    """A fitted scikit-learn forest classifier as per-node arrays: thresholds rounded down to
    float32 (for float32 x, x <= t64 iff x <= the largest float32 not above t64), leaves holding
    the class fractions."""
    from synth import Forest
    trees = est.estimators_ if hasattr(est, "estimators_") else [est]
    offs, feat, thr, left, right, val = [0], [], [], [], [], []
    for tr in trees:
        t = tr.tree_
        t64 = t.threshold.astype(np.float64)
        t32 = t64.astype(np.float32)
        t32 = np.where(t32.astype(np.float64) > t64, np.nextafter(t32, np.float32(-np.inf)), t32)
        leaf = t.children_left < 0
        v = t.value[:, 0, :].astype(np.float64)
        v = v / v.sum(1, keepdims=True)
        feat.append(np.where(leaf, -1, t.feature).astype(np.int32))
        thr.append(np.where(leaf, 0, t32).astype(np.float32))
        left.append(t.children_left.astype(np.int32))
        right.append(t.children_right.astype(np.int32))
        val.append(np.where(leaf[:, None], v, 0).astype(np.float32))
        offs.append(offs[-1] + t.node_count)
    return Forest(n_features=n_features, n_classes=val[0].shape[1],
                  tree_offsets=np.array(offs, np.int64), feature=np.concatenate(feat),
                  threshold=np.concatenate(thr), left=np.concatenate(left),
                  right=np.concatenate(right), value=np.concatenate(val), aggregate=AGG_MEAN)


@pytest.mark.parametrize("kind", ["random", "extra", "single_extra"])
def test_matches_sklearn_forest_classifiers(kind):
    from sklearn.ensemble import ExtraTreesClassifier, RandomForestClassifier
    from sklearn.tree import ExtraTreeClassifier
    rng = np.random.default_rng(5)
    Xt = rng.standard_normal((600, 8)).astype(np.float32)
    yt = (Xt[:, 0] + Xt[:, 1] * Xt[:, 2] > 0).astype(int) + (Xt[:, 3] > 1).astype(int)
    est = {"random": RandomForestClassifier(n_estimators=25, max_depth=9, random_state=0),
           "extra": ExtraTreesClassifier(n_estimators=25, max_depth=9, random_state=0),
           "single_extra": ExtraTreeClassifier(random_state=0)}[kind].fit(Xt, yt)
    f = _from_sklearn(est, 8)
    X = rng.standard_normal((3000, 8)).astype(np.float32)
    X[:300] = Xt[rng.integers(0, 600, 300)]          # rows at the training points
    out, _ = V.predict(f, X)
    ref = est.predict_proba(X)
    assert np.abs(out - ref).max() <= 1e-6
    top2 = np.sort(ref, axis=1)[:, -2:]
    clear = top2[:, 1] - top2[:, 0] > 1e-6
    assert np.array_equal(V.labels(out)[clear], est.predict(X)[clear])


def test_mutations_are_detected():
    rng = np.random.default_rng(2)
    f = with_vector_leaves(random_tiny_forest(rng, 20, 5, max_depth=6), 3, rng)
    X = rng.standard_normal((400, 5)).astype(np.float32)
    out, lv = V.predict(f, X)
    # dividing by the number of classes instead of the number of trees
    wrong = dataclasses.replace(f, aggregate=AGG_SUM)
    s, _ = V.predict(wrong, X)
    assert not np.allclose(s / 3, out)
    assert np.allclose(s / 20, out, rtol=1e-15, atol=1e-15)
    # a leaf vector read at the wrong class offset
    Vr = np.roll(f.value, 1, axis=1)
    r, _ = V.predict(dataclasses.replace(f, value=Vr), X)
    assert not np.allclose(r, out)
