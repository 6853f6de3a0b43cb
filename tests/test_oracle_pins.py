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
