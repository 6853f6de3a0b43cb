"""Randomized differential parity: seeded random forests of many shapes (ragged and perfect,
1-9 features, 1-4 classes, sum/mean, identity/sigmoid/softmax, thresholds on a coarse grid so
ties are common, NaN and infinite inputs, scalar and vector leaves) on every kernel family that
takes them, against the oracles: scores, leaf ids and labels; binned and CSR rows too; wide
rows (global-node kernels) and fused preprocessing as well."""
import dataclasses

import numpy as np
import pytest

import paper_2405_12491_amd as B
from oracle import preprocess as P
from oracle import sparse as S
from oracle import vector as V
from parity_util import assert_leaves, assert_scores, check_labels, oracle_predict, to_dev
from synth import (AGG_MEAN, AGG_SUM, XFORM_IDENTITY, XFORM_SIGMOID, XFORM_SOFTMAX, concat_trees,
                   perfect_tree_arrays, random_tiny_forest, with_vector_leaves)

pytestmark = pytest.mark.gpu

KERNELS = [B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT,
           B.BRIDGER_KERNEL_GEMM]
GRID = np.array([-1.5, -0.5, -0.0, 0.0, 0.25, 0.5, 1.0, 2.0], np.float32)


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _random_case(seed, wide=False):
    """Narrow rows (1-9 features, 1-4 classes), or wide ones (100-900 features, 1-8 classes,
    up to 160 trees: the global-node kernels with lane groups, class slots and 8-class vector
    leaves)."""
    rng = np.random.default_rng((5000 if wide else 1000) + seed)
    F = int(rng.integers(100, 901)) if wide else int(rng.integers(1, 10))
    K = int(rng.integers(1, 9 if wide else 5))
    agg = AGG_MEAN if rng.random() < 0.4 else AGG_SUM
    if K == 1:
        xform = XFORM_SIGMOID if rng.random() < 0.5 else XFORM_IDENTITY
    else:
        xform = XFORM_SOFTMAX if rng.random() < 0.5 else XFORM_IDENTITY
    T = int(rng.integers(K, 160)) if wide else int(rng.integers(K, 3 * K + 20))
    if rng.random() < 0.4:   # perfect trees of one depth
        D = int(rng.integers(1, 9 if wide else 7))
        trees = [perfect_tree_arrays(D, rng.integers(0, F, (1 << D) - 1),
                                     GRID[rng.integers(0, len(GRID), (1 << D) - 1)],
                                     rng.standard_normal(1 << D).astype(np.float32)) for _ in range(T)]
        tc = rng.integers(0, K, T)
        tc[:K] = np.arange(K)
        model = concat_trees(trees, F, K, tc if K > 1 else None, agg, xform,
                             rng.standard_normal(K).astype(np.float32))
    else:
        model = random_tiny_forest(rng, T, F, max_depth=int(rng.integers(1, 11)),
                                   p_split=float(rng.uniform(0.5, 0.9)), thr_grid=GRID,
                                   n_classes=K, aggregate=agg, transform=xform)
        if agg == AGG_MEAN and K > 1:   # every class needs a tree: class of tree t is t mod K
            assert T >= K
    vector = K > 1 and xform != XFORM_SIGMOID and rng.random() < 0.3
    if vector:
        model = with_vector_leaves(model, K, rng, aggregate=agg, transform=xform)
    n = int(rng.integers(1, 400 if wide else 1500))
    X = GRID[rng.integers(0, len(GRID), (n, F))] + (rng.random((n, F)) < 0.3) * rng.standard_normal((n, F))
    X = X.astype(np.float32)
    X[rng.random((n, F)) < 0.02] = np.nan
    X[rng.random((n, F)) < 0.01] = np.inf
    X[rng.random((n, F)) < 0.01] = -np.inf
    return model, X, vector


@pytest.mark.parametrize("seed", range(200))
def test_random_forests(seed):
    _check_case(seed, *_random_case(seed))


@pytest.mark.parametrize("seed", range(60))
def test_random_wide_forests(seed):
    _check_case(f"wide {seed}", *_random_case(seed, wide=True))


@pytest.mark.parametrize("seed", range(40))
def test_random_preprocessed(seed):
    """Random forests behind a random fused preprocessing step (scaler, Binarizer or Normalizer)
    with random parameters; narrow rows for even seeds, wide ones for odd."""
    model, X, vector = _random_case(300 + seed, wide=seed % 2 == 1)
    rng = np.random.default_rng(9000 + seed)
    F = X.shape[1]
    kind = [P.MINMAX, P.CENTER_SCALE, P.BINARIZE, P.NORMALIZE][seed % 4]
    a = b = None
    if kind == P.MINMAX:
        a, b = rng.uniform(-3, 3, F), rng.uniform(-2, 2, F)
    elif kind == P.CENTER_SCALE:
        a, b = rng.standard_normal(F), rng.uniform(0.1, 4, F) * rng.choice([-1, 1], F)
    elif kind == P.BINARIZE:
        a = GRID[rng.integers(0, len(GRID), F)].astype(np.float64)
    _check_case(f"pre {seed}", model, X, vector, (kind, a, b))


# planner overrides (read when a forest is created): every forced shape still passes the
# planner's capacity checks, and a family without a feasible plan reports unsupported
PLAN_OVERRIDES = [("BRIDGER_GLOBAL", ["0", "1"]), ("BRIDGER_ILP", ["1", "2", "4"]),
                  ("BRIDGER_WAVES", ["1", "2", "4", "8"]), ("BRIDGER_ROWS", ["64", "128", "256"]),
                  ("BRIDGER_CHUNK_TREES", ["4", "8", "32"]), ("BRIDGER_NO_FIXED", ["1"])]


@pytest.mark.parametrize("seed", range(40))
def test_random_plans(seed, monkeypatch):
    """Random forests under random launch-shape overrides (global or chunked records, trees
    per lane, waves and rows per workgroup, trees per chunk)."""
    rng = np.random.default_rng(7000 + seed)
    for key, values in PLAN_OVERRIDES:
        if rng.random() < 0.4:
            monkeypatch.setenv(key, str(values[rng.integers(0, len(values))]))
    _check_case(f"plan {seed}", *_random_case(600 + seed, wide=seed % 3 == 2))


def _check_case(seed, model, X, vector, pre=None):
    import torch
    Xp = X if pre is None else P.apply(pre[0], pre[1], pre[2], X)
    if vector:
        ref, ref_lv = V.predict(model, Xp)
    else:
        ref, ref_lv = oracle_predict(model, Xp, leaves=True)
    Xd = to_dev(X)
    K = model.n_classes
    classifier = K > 1 or model.transform == XFORM_SIGMOID
    with B.Forest(model) as f:
        if pre is not None:
            f.set_preprocess(*pre)
        ran = 0
        for k in KERNELS:
            try:
                f.kernel = k
            except B.BridgerError as e:
                assert e.status == B.BRIDGER_ERR_UNSUPPORTED
                continue
            what = f"seed {seed} {B.KERNEL_NAMES[k]}"
            out = f.predict(Xd)
            lv = f.predict_leaves(Xd)
            lab = f.predict_labels(Xd) if classifier else None
            torch.cuda.synchronize()
            assert_scores(out.cpu().numpy(), ref, what + " scores")
            assert_leaves(lv.cpu().numpy(), ref_lv, what + " leaves")
            if classifier:
                check_labels(lab.cpu().numpy(), ref, what + " labels")
            ran += 1
        assert ran >= 1
        f.kernel = B.BRIDGER_KERNEL_AUTO
        if f.kernel in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
            if f.bin_info()["bin_bytes"]:
                q = f.bin(Xd)
                try:
                    out = f.predict_binned(q)
                except B.BridgerError as e:  # a forced shape can leave the bins no plan
                    assert e.status == B.BRIDGER_ERR_UNSUPPORTED and "plan" in str(seed)
                else:
                    torch.cuda.synchronize()
                    assert_scores(out.cpu().numpy(), ref, f"seed {seed} binned")
            nz = np.nonzero(np.where(np.isnan(X), 1.0, X))
            ip = np.concatenate([[0], np.cumsum(np.bincount(nz[0], minlength=X.shape[0]))]).astype(np.int64)
            d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
            out = f.predict_csr(d(ip), d(nz[1].astype(np.int32)), d(X[nz].astype(np.float32)), X.shape[0])
            torch.cuda.synchronize()
            assert_scores(out.cpu().numpy(), ref, f"seed {seed} csr")
