"""The oracle against what the mathematics fixes, and proof that the pins bite.

The mutation tests compile deliberately broken copies of the oracle (a plausible
mistake each: a flipped tie rule, NaN sent left, swapped children, a dropped tree,
a wrong class or row index, a lost base score, a wrong mean divisor, a sign error in
the logistic function, a dropped softmax term) and require that at least one pin
rejects every one of them.
"""
import os
import subprocess
import tempfile

import numpy as np
import pytest

import oracle
import oracle_pins as P

pytestmark = pytest.mark.cpu


@pytest.fixture(scope="module")
def lib():
    oracle.build()
    return oracle.load()


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(lib, pin):
    pin(lib)


SRC = open(os.path.join(os.path.dirname(oracle.__file__), "forest_oracle.c")).read()

MUTANTS = {
    "tie_goes_right": ("double)left[n] : (int64_t)right[n];", None, "(xv <= tv)", "(xv < tv)"),
    "nan_goes_left": (None, None, "(xv <= tv)", "!(xv > tv)"),
    "children_swapped": (None, None, "? (int64_t)left[n] : (int64_t)right[n]", "? (int64_t)right[n] : (int64_t)left[n]"),
    "last_tree_dropped": (None, None, "for (int32_t t = 0; t < n_trees; ++t) {\n      int64_t a", "for (int32_t t = 0; t < n_trees - 1; ++t) {\n      int64_t a"),
    "class_map_ignored": (None, None, "int32_t k = tree_class ? tree_class[t] : t % n_classes;\n      acc[k]", "int32_t k = tree_class ? tree_class[t] : 0;\n      acc[k]"),
    "row_stride": (None, None, "const float *x = X + r * (int64_t)n_features;", "const float *x = X + r;"),
    "base_dropped": (None, None, "acc[k] = (aggregate == 0 && base_score) ? (double)base_score[k] : 0.0;", "acc[k] = 0.0;"),
    "mean_over_all_trees": (None, None, "base + acc[k] / (double)count[k]", "base + acc[k] / (double)n_trees"),
    "sigmoid_sign": (None, None, "return 1.0 / (1.0 + exp(-z));", "return 1.0 / (1.0 + exp(z));"),
    "softmax_term_dropped": (None, None, "z[k] = exp(z[k] - m); s += z[k];", "z[k] = exp(z[k] - m); if (k) s += z[k];"),
    "feature_from_wrong_node": (None, None, "double xv = (double)x[f];", "double xv = (double)x[(f + 1) % n_features];"),
    "leaf_value_index": (None, None, "acc[k] + (double)value[a + leaf];", "acc[k] + (double)value[a + leaf - 1 + (leaf == 0)];"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name):
    _, _, old, new = MUTANTS[name]
    assert SRC.count(old) == 1, f"mutation anchor for {name} not unique"
    src = SRC.replace(old, new)
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "m.c")
        so = os.path.join(d, "m.so")
        open(c, "w").write(src)
        oracle.build(c, so)
        lib = oracle.load(so)
        caught = []
        for pin in P.ALL_PINS:
            try:
                pin(lib)
            except (AssertionError, oracle.OracleError, IndexError, ValueError) as e:  # noqa: PERF203
                caught.append((pin.__name__, type(e).__name__))
        assert caught, f"no pin rejects mutant {name}"


@pytest.mark.parametrize("name,n", [("gbdt_d6", 1003), ("mc_gbdt_d8", 353), ("ragged_d12", 351)])
def test_oracle_thread_split(name, n):
    """The wrapper's row split over threads: 7 threads on a row count that 7 does not divide
    give the one-thread results bit for bit (scores and leaf ids), and both agree with the
    independent vectorized traversal on every leaf id."""
    from synth import make_workload
    assert n % 7 != 0
    w = make_workload(name, n)
    X = w.X()
    o1, l1, v1 = oracle.predict(w.forest, X, want_leaves=True, threads=1)
    o7, l7, v7 = oracle.predict(w.forest, X, want_leaves=True, threads=7)
    assert np.array_equal(o1, o7) and np.array_equal(l1, l7) and v1 == v7
    _, lv = P.numpy_traverse(w.forest, X)
    assert np.array_equal(l7, lv)
