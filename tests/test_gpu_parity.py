"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Leaf ids must match bit for bit; scores within 1e-6 + 1e-5 * |oracle|.  Every kernel family
that can run a forest is checked on it.  Sizes span several row tiles plus a ragged tail.
"""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import (assert_leaves, assert_scores, check_parity, gpu_predict, oracle_predict,
                         to_dev)
from synth import (AGG_MEAN, AGG_SUM, CONFIGS, XFORM_IDENTITY, XFORM_SIGMOID, XFORM_SOFTMAX,
                   concat_trees, make_workload, perfect_tree_arrays, permute_nodes,
                   random_tiny_forest)

pytestmark = pytest.mark.gpu

KERNELS = [B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT,
           B.BRIDGER_KERNEL_GEMM]

# rows per workload for the oracle-sized cases: several tiles of the largest row tile (1024)
# plus a tail that is not a multiple of 32
SMALL_ROWS = {"dt_d3": 10_000, "rf_d8": 3 * 1024 + 77, "gbdt_d6": 3 * 1024 + 77,
              "mc_gbdt_d8": 2 * 32 * 3 + 45, "ragged_d12": 3 * 64 + 29}


def supported(f: B.Forest, k: int) -> bool:
    try:
        f.kernel = k
        return True
    except B.BridgerError as e:
        assert e.status == B.BRIDGER_ERR_UNSUPPORTED
        return False


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


@pytest.mark.parametrize("name", list(CONFIGS))
def test_workload_small(name):
    w = make_workload(name, SMALL_ROWS[name])
    X = w.X()
    Xd = to_dev(X)
    ran = 0
    with B.Forest(w.forest) as f:
        for k in KERNELS:
            if not supported(f, k):
                continue
            print(f"[parity] {name} rows={X.shape[0]} kernel={B.KERNEL_NAMES[k]}", flush=True)
            check_parity(w.forest, X, k, f"{name}/{B.KERNEL_NAMES[k]}", Xd=Xd, forest=f)
            ran += 1
    assert ran >= 2


@pytest.mark.parametrize("name", ["shallow_d3", "shallow_d4"])
def test_shallow_workloads_all_kernels(name):
    """The matrix-multiply lowering and the traversal kernels on shallow forests."""
    w = make_workload(name, 3 * 1024 + 77)
    X = w.X()
    X[5, 3] = np.nan                     # rows with non-finite features take the walk fallback
    X[17, 0] = np.inf
    X[700, 27] = -np.inf
    Xd = to_dev(X)
    with B.Forest(w.forest) as f:
        assert supported(f, B.BRIDGER_KERNEL_GEMM)
        for k in KERNELS:
            if supported(f, k):
                check_parity(w.forest, X, k, f"{name}/{B.KERNEL_NAMES[k]}", Xd=Xd, forest=f)


def test_direct_sums_bit_identical():
    """One row per lane, trees in ascending order: the double-precision sum is the oracle's."""
    for name in ("dt_d3", "rf_d8", "ragged_d12"):
        w = make_workload(name, 500)
        X = w.X()
        check_parity(w.forest, X, B.BRIDGER_KERNEL_DIRECT, name + "/direct", exact_sum=True)


def test_perfect_single_group_sums_bit_identical():
    w = make_workload("rf_d8", 2048 + 5)
    X = w.X()
    check_parity(w.forest, X, B.BRIDGER_KERNEL_PERFECT, "rf_d8/perfect", exact_sum=True)


@pytest.mark.parametrize("n", [1, 2, 31, 32, 33, 63, 64, 65, 255, 257, 1023, 1025])
def test_row_counts(n):
    w = make_workload("gbdt_d6", n)
    X = w.X()
    with B.Forest(w.forest) as f:
        for k in KERNELS:
            if supported(f, k):
                check_parity(w.forest, X, k, f"gbdt_d6 n={n} {B.KERNEL_NAMES[k]}", forest=f)


def test_zero_rows_launches_nothing():
    import torch
    w = make_workload("gbdt_d6", 4)
    with B.Forest(w.forest) as f:
        X = torch.zeros((0, 28), device="cuda")
        out = torch.full((0, 1), 7.0, device="cuda")
        f.predict(X, out)
        torch.cuda.synchronize()


FLT_MAX = np.float32(3.4028235e38)


def _adversarial_rows(F, thr_values, rng, n=600):
    X = rng.standard_normal((n, F)).astype(np.float32)
    specials = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0, 1e-45, -1e-45, 1.17549435e-38,
                         FLT_MAX, -FLT_MAX], np.float32)
    m = rng.random(X.shape) < 0.15
    X[m] = specials[rng.integers(0, len(specials), m.sum())]
    t = np.asarray(thr_values, np.float32)
    m = rng.random(X.shape) < 0.25
    pick = t[rng.integers(0, len(t), m.sum())]
    nudge = rng.integers(-1, 2, m.sum())
    vals = np.where(nudge == 0, pick, np.where(nudge > 0, np.nextafter(pick, np.float32(np.inf)),
                                               np.nextafter(pick, np.float32(-np.inf))))
    X[m] = vals.astype(np.float32)
    return X


# thresholds on zero of either sign, denormals and the largest finite values; the second grid
# adds infinite thresholds, which switch the perfect kernel from its sign-of-difference step
# to the plain compare
THRESHOLD_GRIDS = {
    "finite": [-1.0, -1e-45, -0.0, 0.0, 1e-45, 0.5, 2.0, FLT_MAX, -FLT_MAX],
    "with_inf": [-1.0, -0.0, 0.0, 1e-45, 0.5, np.inf, -np.inf, FLT_MAX],
}


@pytest.mark.parametrize("grid_name", list(THRESHOLD_GRIDS))
@pytest.mark.parametrize("F", [3, 7, 28])
def test_adversarial_values(F, grid_name, monkeypatch):
    """NaN, +-inf, +-0, denormals, +-FLT_MAX, values on a threshold and one ulp either side."""
    rng = np.random.default_rng(100 + F)
    grid = np.array(THRESHOLD_GRIDS[grid_name], np.float32)
    G = len(grid)
    trees = []
    for D in (2, 3, 4, 5):
        for _ in range(3):
            n_int = (1 << D) - 1
            trees.append(perfect_tree_arrays(D, rng.integers(0, F, n_int), grid[rng.integers(0, G, n_int)],
                                             rng.standard_normal(1 << D).astype(np.float32)))
    ragged = concat_trees(trees, F)
    perfect = concat_trees([perfect_tree_arrays(4, rng.integers(0, F, 15), grid[rng.integers(0, G, 15)],
                                                rng.standard_normal(16).astype(np.float32))
                            for _ in range(9)], F)
    X = _adversarial_rows(F, grid, rng)
    for model in (ragged, perfect):
        for sign_step in ("on", "off"):
            # the variable is read when the forest is created
            if sign_step == "off":
                monkeypatch.setenv("BRIDGER_NO_SIGN_STEP", "1")
            else:
                monkeypatch.delenv("BRIDGER_NO_SIGN_STEP", raising=False)
            with B.Forest(model) as f:
                for k in KERNELS:
                    if supported(f, k):
                        check_parity(model, X, k, f"adversarial F={F} {grid_name} sign_step={sign_step} "
                                     f"{B.KERNEL_NAMES[k]}", forest=f)


@pytest.mark.parametrize("deep", ["1", "0"])
@pytest.mark.parametrize("grid_name", list(THRESHOLD_GRIDS))
@pytest.mark.parametrize("F", [7, 28])
def test_adversarial_values_global(F, grid_name, deep, monkeypatch):
    """The same values through the global-node perfect kernel (top levels from LDS copies),
    with and without the deep blocks: both level steps (finite thresholds: sign of the
    difference; infinite ones: compare) on depths whose deep levels end in a block with leaf
    values (4, 8) and in a leaf array (5, 7)."""
    monkeypatch.setenv("BRIDGER_GLOBAL", "1")
    monkeypatch.setenv("BRIDGER_DEEP", deep)
    rng = np.random.default_rng(200 + F)
    grid = np.array(THRESHOLD_GRIDS[grid_name], np.float32)
    for D in (4, 5, 7, 8):
        n_int = (1 << D) - 1
        model = concat_trees([perfect_tree_arrays(D, rng.integers(0, F, n_int),
                                                  grid[rng.integers(0, len(grid), n_int)],
                                                  rng.standard_normal(1 << D).astype(np.float32))
                              for _ in range(9)], F)
        X = _adversarial_rows(F, grid, rng, n=700)
        with B.Forest(model) as f:
            print(f"[adversarial-global] F={F} D={D} {grid_name} deep={deep} "
                  f"plan={f.plan(X.shape[0])}", flush=True)
            check_parity(model, X, B.BRIDGER_KERNEL_PERFECT,
                         f"adversarial global F={F} D={D} {grid_name} deep={deep}", forest=f)


def test_unaligned_rows():
    """X starting 4 bytes past a 16-byte boundary takes the scalar row-load path."""
    import torch
    w = make_workload("gbdt_d6", 700)
    X = w.X()
    big = torch.zeros(X.size + 1, dtype=torch.float32, device="cuda")
    big[1:] = torch.from_numpy(X.reshape(-1)).cuda()
    Xd = big[1:].view(X.shape)
    assert Xd.data_ptr() % 16 == 4
    with B.Forest(w.forest) as f:
        for k in KERNELS:
            if supported(f, k):
                check_parity(w.forest, X, k, f"unaligned {B.KERNEL_NAMES[k]}", Xd=Xd, forest=f)


def test_permuted_numbering_and_leaf_map():
    """Caller node ids in random order: leaf ids come back in the caller's numbering."""
    rng = np.random.default_rng(7)
    w = make_workload("rf_d8", 900)
    model = permute_nodes(w.forest, rng)
    X = w.X()
    with B.Forest(model) as f:
        for k in KERNELS:
            if supported(f, k):
                check_parity(model, X, k, f"permuted {B.KERNEL_NAMES[k]}", forest=f)


@pytest.mark.parametrize("n_trees", [1, 2, 3, 5, 33])
def test_tree_counts_and_shapes(n_trees):
    rng = np.random.default_rng(n_trees)
    model = random_tiny_forest(rng, n_trees, 9, max_depth=9, p_split=0.75)
    X = rng.standard_normal((333, 9)).astype(np.float32)
    with B.Forest(model) as f:
        for k in KERNELS:
            if supported(f, k):
                check_parity(model, X, k, f"T={n_trees} {B.KERNEL_NAMES[k]}", forest=f)
    # perfect trees too
    trees = [perfect_tree_arrays(3, rng.integers(0, 9, 7), rng.standard_normal(7).astype(np.float32),
                                 rng.standard_normal(8).astype(np.float32)) for _ in range(n_trees)]
    model = concat_trees(trees, 9)
    with B.Forest(model) as f:
        for k in KERNELS:
            if supported(f, k):
                check_parity(model, X, k, f"perfect T={n_trees} {B.KERNEL_NAMES[k]}", forest=f)


def test_depth_zero_trees():
    rng = np.random.default_rng(3)
    stump = perfect_tree_arrays(1, np.array([2]), np.array([0.0], np.float32), np.array([-1.0, 1.0], np.float32))
    leaf = (np.array([-1], np.int32), np.zeros(1, np.float32), np.array([-1], np.int32),
            np.array([-1], np.int32), np.array([2.5], np.float32))
    model = concat_trees([leaf, stump, leaf, leaf, stump], 4)
    X = rng.standard_normal((200, 4)).astype(np.float32)
    with B.Forest(model) as f:
        for k in KERNELS:
            if supported(f, k):
                check_parity(model, X, k, f"depth0 {B.KERNEL_NAMES[k]}", forest=f)


@pytest.mark.parametrize("agg,xform,K", [(AGG_SUM, XFORM_SOFTMAX, 3), (AGG_MEAN, XFORM_IDENTITY, 4),
                                         (AGG_MEAN, XFORM_SOFTMAX, 5), (AGG_SUM, XFORM_SIGMOID, 1),
                                         (AGG_MEAN, XFORM_SIGMOID, 1)])
def test_classes_aggregates_transforms(agg, xform, K):
    rng = np.random.default_rng(K * 10 + agg)
    T = 23
    trees = [perfect_tree_arrays(4, rng.integers(0, 6, 15), rng.standard_normal(15).astype(np.float32),
                                 rng.standard_normal(16).astype(np.float32)) for _ in range(T)]
    tc = rng.integers(0, K, T)
    tc[:K] = np.arange(K)  # every class has a tree
    base = rng.standard_normal(K).astype(np.float32)
    X = rng.standard_normal((1100, 6)).astype(np.float32)
    for model in (concat_trees(trees, 6, K, tc, agg, xform, base),
                  permute_nodes(concat_trees(trees, 6, K, None, agg, xform, base), rng)):
        with B.Forest(model) as f:
            for k in KERNELS:
                if supported(f, k):
                    check_parity(model, X, k, f"K={K} agg={agg} x={xform} {B.KERNEL_NAMES[k]}", forest=f)


# launch shapes and kernel variants the planner does not pick for these forests, forced with
# the planner's tuning variables (read when a forest is created)
VARIANT_ENVS = [
    {"BRIDGER_GLOBAL": "1"},                                   # records from global memory
    {"BRIDGER_GLOBAL": "1", "BRIDGER_NO_SIGN_STEP": "1"},      # (top 3 levels from LDS copies)
    {"BRIDGER_GLOBAL": "1", "BRIDGER_PERFECT_TOP_LEVELS": "3"},  # top 3 levels, 16 trees a lane
    {"BRIDGER_GLOBAL": "1", "BRIDGER_PERFECT_TOP_LEVELS": "5"},  # top 5 levels, 8 trees (2 KB)
    {"BRIDGER_GLOBAL": "1", "BRIDGER_TOP_GROUP_KB": "2"},      # top 4 levels, 16 trees (2 KB)
    {"BRIDGER_GLOBAL": "1", "BRIDGER_REG_SUMS": "0"},          # class sums in LDS
    {"BRIDGER_GLOBAL": "1", "BRIDGER_TOPS": "0"},              # every level from global memory
    {"BRIDGER_GLOBAL": "1", "BRIDGER_DEEP": "0"},              # top levels, then one record a level
    {"BRIDGER_GLOBAL": "1", "BRIDGER_WAVES": "8", "BRIDGER_ROWS": "32"},    # 2 groups a wave
    {"BRIDGER_GLOBAL": "1", "BRIDGER_WAVES": "8", "BRIDGER_ROWS": "128"},   # groups of 2 waves
    {"BRIDGER_NO_FIXED": "1"},                                 # run-time chunk geometry
    {"BRIDGER_SIZED_PLANS": "0"},                              # the large-batch plan on small n
    {"BRIDGER_CHUNK_TREES": "4"},                              # compile-time chunks of 4, 8, 32
    {"BRIDGER_CHUNK_TREES": "8"},
    {"BRIDGER_CHUNK_TREES": "32"},
    {"BRIDGER_ILP": "1", "BRIDGER_WAVES": "4", "BRIDGER_ROWS": "64"},   # 4 lane groups, 1 tree
    {"BRIDGER_ILP": "2", "BRIDGER_WAVES": "2", "BRIDGER_ROWS": "64"},   # 2 lane groups, 2 trees
    {"BRIDGER_ILP": "4", "BRIDGER_WAVES": "4", "BRIDGER_ROWS": "64"},   # 4 lane groups, 4 trees:
]                                                                      # class sums in registers


def _variant_models():
    rng = np.random.default_rng(77)
    K, T = 3, 23
    trees = [perfect_tree_arrays(4, rng.integers(0, 6, 15), rng.standard_normal(15).astype(np.float32),
                                 rng.standard_normal(16).astype(np.float32)) for _ in range(T)]
    tc = rng.integers(0, K, T)
    tc[:K] = np.arange(K)
    multi = concat_trees(trees, 6, K, tc, AGG_SUM, XFORM_SOFTMAX, rng.standard_normal(K).astype(np.float32))
    X6 = rng.standard_normal((1100, 6)).astype(np.float32)
    g = make_workload("gbdt_d6", 1500)
    r = make_workload("rf_d8", 700)
    import dataclasses
    g3 = dataclasses.replace(g.forest, n_classes=3, aggregate=AGG_MEAN, transform=XFORM_SOFTMAX,
                             tree_class=(np.arange(g.forest.n_trees) % 3).astype(np.int32),
                             base_score=rng.standard_normal(3).astype(np.float32))
    return [("gbdt_d6", g.forest, g.X()), ("rf_d8", r.forest, r.X()), ("multiclass", multi, X6),
            ("multiclass28", g3, g.X())]


@pytest.mark.parametrize("env", [{"BRIDGER_GLOBAL": "1"}, {"BRIDGER_GLOBAL": "1", "BRIDGER_ILP": "2"},
                                 {"BRIDGER_GLOBAL": "1", "BRIDGER_ILP": "4"}, {"BRIDGER_GLOBAL": "0"},
                                 {"BRIDGER_TOPS": "0"}, {"BRIDGER_TREELETS": "0"},
                                 {"BRIDGER_TREELETS": "0", "BRIDGER_TOP_LEVELS": "4"},
                                 {"BRIDGER_TREELETS": "0", "BRIDGER_TOP_LEVELS": "4", "BRIDGER_ROWS": "128"},
                                 {"BRIDGER_ROWS": "256", "BRIDGER_WAVES": "8"},
                                 {"BRIDGER_TREELETS": "0", "BRIDGER_ROWS": "256", "BRIDGER_WAVES": "8"},
                                 {"BRIDGER_COALESCED_TILE": "0"},
                                 {"BRIDGER_TREELET_LDS_LEVELS": "2"},
                                 {"BRIDGER_TREELET_LDS_LEVELS": "2", "BRIDGER_ROWS": "256", "BRIDGER_WAVES": "8"}],
                         ids=lambda e: ",".join(f"{k[8:]}={v}" for k, v in e.items()))
def test_ragged_kernel_variants(env, monkeypatch):
    """The ragged kernel with records in LDS chunks and read from global memory (one or two
    runs per lane; two-level treelets, or the top levels from per-wave LDS copies of 4 or 5
    levels, with lane groups of one, two or four waves, or without them), on ragged,
    multiclass and leaf-id cases."""
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    rng = np.random.default_rng(91)
    models = []
    w = make_workload("ragged_d12", 3 * 64 + 29)
    models.append(("ragged_d12", w.forest, w.X()))
    rf = random_tiny_forest(rng, 40, 6, max_depth=9)
    X6 = rng.standard_normal((700, 6)).astype(np.float32)
    models.append(("tiny_ragged", rf, X6))
    multi = random_tiny_forest(rng, 40, 6, max_depth=9, n_classes=3, aggregate=AGG_MEAN,
                               transform=XFORM_SOFTMAX)
    models.append(("multiclass_ragged", multi, X6))
    for name, model, X in models:
        with B.Forest(model) as f:
            if not supported(f, B.BRIDGER_KERNEL_RAGGED):
                continue
            print(f"[variant] {env} {name} plan={f.plan(X.shape[0])}", flush=True)
            check_parity(model, X, B.BRIDGER_KERNEL_RAGGED, f"{name} {env}", forest=f)


def _class_layouts(T, rng):
    """Class assignments that stress the global kernels' class slots (a lane group's tree
    range is contiguous in class order): empty classes, one-tree classes next to classes
    spread over several groups, classes given in shuffled tree order, and groups whose trees
    span more classes (empty ones between) than the kernels' small register class slots hold."""
    K1 = 7
    tc1 = np.array([0] * 20 + [1] + [3] * 2 + [4] * 30 + [6] * (T - 53))  # 2 and 5 empty
    K2 = 12
    tc2 = np.arange(T) % K2                                                # interleaved
    K3 = 3
    tc3 = np.r_[np.zeros(T - 2, int), [1, 2]]                              # one huge class
    K4 = 16
    tc4 = np.repeat([0, 5, 10, 15], [14, 18, 15, T - 47])                  # spans of 6 classes
    # with 16 groups of 4 trees: the widest group spans exactly 4 classes (the small slot
    # count), or exactly 5, with an empty class inside (the large one)
    K5 = 5
    tc5 = np.array([0] * 4 + [1, 2, 3, 4] + [4] * (T - 8))
    K6 = 9
    tc6 = np.array([0] * 4 + [1, 2, 3, 4] + [4] * 4 + [4, 6, 7, 8] + [8] * (T - 16))
    return [(K1, rng.permutation(tc1)), (K2, tc2), (K3, tc3), (K4, tc4), (K5, tc5), (K6, tc6)]


@pytest.mark.parametrize("family", ["perfect", "ragged"])
@pytest.mark.parametrize("env", [{"BRIDGER_GLOBAL": "1", "BRIDGER_WAVES": "16", "BRIDGER_ROWS": "64"},
                                 {"BRIDGER_GLOBAL": "1", "BRIDGER_WAVES": "8", "BRIDGER_ROWS": "32"}],
                         ids=lambda e: ",".join(f"{k[8:]}={v}" for k, v in e.items()))
def test_global_class_slots(family, env, monkeypatch):
    """Global-node kernels with 16 lane groups on several classes: each group sums the classes
    its contiguous tree range touches, the groups' partials are added in group order; SUM
    (with empty classes: base score only) and MEAN (every class non-empty), softmax and
    identity."""
    import dataclasses
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    rng = np.random.default_rng(2024)
    T, F = 64, 9
    X = rng.standard_normal((3 * 64 + 29, F)).astype(np.float32)
    if family == "perfect":
        trees = [perfect_tree_arrays(5, rng.integers(0, F, 31), rng.standard_normal(31).astype(np.float32),
                                     rng.standard_normal(32).astype(np.float32)) for _ in range(T)]
        base_model = concat_trees(trees, F)
        kernel = B.BRIDGER_KERNEL_PERFECT
    else:
        base_model = random_tiny_forest(rng, T, F, max_depth=9)
        kernel = B.BRIDGER_KERNEL_RAGGED
    for K, tc in _class_layouts(T, rng):
        empty = len(np.unique(tc)) < K
        for agg, xform in ((AGG_SUM, XFORM_SOFTMAX), (AGG_MEAN, XFORM_IDENTITY)):
            if agg == AGG_MEAN and empty:
                continue  # MEAN over an empty class is rejected at create
            model = dataclasses.replace(base_model, n_classes=K, tree_class=np.asarray(tc, np.int32),
                                        aggregate=agg, transform=xform,
                                        base_score=rng.standard_normal(K).astype(np.float32))
            with B.Forest(model) as f:
                if not supported(f, kernel):
                    continue
                p = f.plan(X.shape[0])
                print(f"[slots] {family} {env} K={K} agg={agg} plan={p}", flush=True)
                R = int(env["BRIDGER_ROWS"])
                G = 64 * int(env["BRIDGER_WAVES"]) // R
                # the global-node plan: the row tile and G x K class slots per row, plus the
                # waves' top-level copies when the plan uses them (perfect: 1 KB per lane group
                # of every wave; ragged with one class: 1 KB per wave, which holds the sums)
                W = int(env["BRIDGER_WAVES"])
                assert p["rows_per_wg"] == R and p["chunk_bytes"] == 0
                tile, slots = F * R * 4, G * K * R * 8
                if family == "perfect":
                    # class sums in LDS, or (deep blocks, at most 16 classes) in registers and
                    # written into the tile after the walk; copies of 1 or 2 KB per lane group
                    copies = [W * max(1, 64 // R) * kb for kb in (1024, 2048)]
                    allowed = (tile + slots,) + tuple(tile + slots + c for c in copies) + \
                        tuple(tile + c for c in copies)
                else:
                    allowed = (tile + slots,) + ((tile + W * 1024,) if K == 1 and R >= 64 else ())
                assert p["lds_bytes"] in allowed, (p["lds_bytes"], allowed)
                check_parity(model, X, kernel, f"{family} K={K} agg={agg} {env}", forest=f)


@pytest.mark.parametrize("env", VARIANT_ENVS, ids=lambda e: ",".join(f"{k[8:]}={v}" for k, v in e.items()))
def test_perfect_kernel_variants(env, monkeypatch):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    for name, model, X in _variant_models():
        with B.Forest(model) as f:
            if not supported(f, B.BRIDGER_KERNEL_PERFECT):
                continue
            print(f"[variant] {env} {name} plan={f.plan(X.shape[0])}", flush=True)
            check_parity(model, X, B.BRIDGER_KERNEL_PERFECT, f"{name} {env}", forest=f)


# batch sizes in each of the planner's size classes (up to 8192, 32768, 131072 and 524288 rows;
# larger batches take the large-batch plan)
SIZE_CLASS_ROWS = [1, 325, 5000, 20000, 100000]


def _size_class_models():
    from synth import with_vector_leaves
    rng = np.random.default_rng(91)
    F, T = 9, 22
    trees = [perfect_tree_arrays(6, rng.integers(0, F, 63), rng.standard_normal(63).astype(np.float32),
                                 rng.standard_normal(64).astype(np.float32)) for _ in range(T)]
    one = concat_trees(trees, F, 1, None, AGG_SUM, XFORM_SIGMOID, np.zeros(1, np.float32))
    tc = np.arange(T) % 3
    multi = concat_trees(trees, F, 3, tc, AGG_SUM, XFORM_SOFTMAX, rng.standard_normal(3).astype(np.float32))
    models = [("K=1", one), ("K=3", multi)]
    for K in (2, 3, 8):
        models.append((f"vector K={K}", with_vector_leaves(one, K, rng, AGG_MEAN, XFORM_SOFTMAX)))
    X = rng.standard_normal((max(SIZE_CLASS_ROWS), F)).astype(np.float32)
    return models, X


def test_batch_size_classes():
    """Every batch-size class's plan (each with its own row tile and traversal copy) against
    the oracle, for scalar and vector leaves, on fp32 rows and on bins."""
    import torch
    models, X = _size_class_models()
    Xd = to_dev(X)
    from oracle import vector as V
    for name, model in models:
        if np.ndim(model.value) == 2:
            ref, ref_lv = V.predict(model, X, threads=8)
        else:
            ref, ref_lv = oracle_predict(model, X, leaves=True)
        with B.Forest(model) as f:
            f.kernel = B.BRIDGER_KERNEL_PERFECT
            q = f.bin(Xd)
            plans = set()
            for n in SIZE_CLASS_ROWS:
                p = f.plan(n)
                plans.add((p["rows_per_wg"], p["chunk_bytes"], p["lds_bytes"]))
                print(f"[sized] {name} n={n} plan={p}", flush=True)
                what = f"{name} n={n}"
                assert_scores(gpu_predict(f, Xd[:n]), ref[:n], what + " scores")
                assert_leaves(gpu_predict(f, Xd[:n], leaves=True), ref_lv[:n], what + " leaves")
                out = f.predict_binned(q[:n])
                lv = f.predict_binned_leaves(q[:n])
                torch.cuda.synchronize()
                assert_scores(out.cpu().numpy().astype(np.float64), ref[:n], what + " binned scores")
                assert_leaves(lv.cpu().numpy(), ref_lv[:n], what + " binned leaves")
            # small batches get plans of their own (more, smaller workgroups)
            assert len(plans) >= 2, (name, plans)


def test_determinism_and_streams():
    import torch
    w = make_workload("gbdt_d6", 5000)
    Xd = to_dev(w.X())
    with B.Forest(w.forest) as f:
        a = gpu_predict(f, Xd)
        b = gpu_predict(f, Xd)
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            out = f.predict(Xd)
        s.synchronize()
        c = out.cpu().numpy()
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(a.view(np.uint32), c.view(np.uint32))


def test_concurrent_host_threads():
    """One handle serving several host threads at once, each with its own stream and rows (the
    C calls release the interpreter lock): every thread's scores, leaf ids and binned scores
    match the single-threaded results bit for bit, over repeated rounds."""
    import threading
    import torch
    w = make_workload("gbdt_d6", 4000)
    Xs = [to_dev((w.X() * np.float32(1 + 0.25 * i)).astype(np.float32)) for i in range(4)]
    with B.Forest(w.forest) as f:
        want = []
        for Xd in Xs:
            want.append((gpu_predict(f, Xd), gpu_predict(f, Xd, leaves=True),
                         f.predict_binned(f.bin(Xd)).cpu().numpy()))
        errors = []

        def worker(i):
            try:
                s = torch.cuda.Stream()
                with torch.cuda.stream(s):
                    for _ in range(20):
                        out = f.predict(Xs[i])
                        lv = f.predict_leaves(Xs[i])
                        ob = f.predict_binned(f.bin(Xs[i]))
                    s.synchronize()
                assert np.array_equal(out.cpu().numpy().view(np.uint32), want[i][0].view(np.uint32))
                assert np.array_equal(lv.cpu().numpy(), want[i][1])
                assert np.array_equal(ob.cpu().numpy().view(np.uint32), want[i][2].view(np.uint32))
            except Exception as e:  # reported on the main thread
                errors.append((i, repr(e)))

        threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
        for t in threads:
            t.start()
        for t in threads:
            t.join()
        assert not errors, errors


def test_argument_errors():
    import torch
    w = make_workload("gbdt_d6", 64)
    Xd = to_dev(w.X())
    with B.Forest(w.forest) as f:
        out = torch.empty((64, 1), device="cuda")
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_predict(f.handle, Xd.data_ptr(), 64, 27, out.data_ptr(), 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_predict(f.handle, Xd.data_ptr(), 64, 28, Xd.data_ptr() + 64, 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_predict(f.handle, Xd.data_ptr(), -1, 28, out.data_ptr(), 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT


# The full-size workloads are checked exhaustively (every score, every leaf id) in
# test_gpu_full_parity.py.


def _chain_tree(depth, F, rng):
    """A tree of the given depth shaped as a chain: internal node k (id 2k) has a leaf on its
    left (id 2k + 1) and internal node k + 1 on its right; the last right child is a leaf.
    Most thresholds are low, so most rows run deep; every eighth is 0.0."""
    n = 2 * depth + 1
    feat = np.full(n, -1, np.int32)
    thr = np.zeros(n, np.float32)
    left = np.full(n, -1, np.int32)
    right = np.full(n, -1, np.int32)
    val = rng.standard_normal(n).astype(np.float32)
    for k in range(depth):
        feat[2 * k] = k % F
        thr[2 * k] = 0.0 if k % 8 == 7 else -5.0
        left[2 * k], right[2 * k] = 2 * k + 1, 2 * k + 2
        val[2 * k] = 0.0
    return feat, thr, left, right, val


def test_maximum_sizes():
    """Limits: 64 classes; a depth-64 tree; perfect trees of depth 10 (the PERFECT limit) and 11;
    rows of 5,000 features (no LDS plan fits: the DIRECT fallback)."""
    rng = np.random.default_rng(64)
    X12 = rng.standard_normal((777, 12)).astype(np.float32)
    cases = []
    T = 128
    trees = [perfect_tree_arrays(3, rng.integers(0, 12, 7), rng.standard_normal(7).astype(np.float32),
                                 rng.standard_normal(8).astype(np.float32)) for _ in range(T)]
    cases.append(("64 classes", concat_trees(trees, 12, 64, np.arange(T) % 64, AGG_SUM, XFORM_SOFTMAX,
                                             rng.standard_normal(64).astype(np.float32)), X12))
    deep = [_chain_tree(64, 12, rng), _chain_tree(40, 12, rng)]
    cases.append(("depth 64", concat_trees(deep, 12), X12))
    for D in (10, 11):
        n_int = (1 << D) - 1
        trees = [perfect_tree_arrays(D, rng.integers(0, 12, n_int),
                                     rng.standard_normal(n_int).astype(np.float32),
                                     rng.standard_normal(n_int + 1).astype(np.float32))
                 for _ in range(2)]
        cases.append((f"perfect depth {D}", concat_trees(trees, 12), X12))
    wide = random_tiny_forest(rng, 12, 5000, max_depth=6)
    cases.append(("5000 features", wide, rng.standard_normal((300, 5000)).astype(np.float32)))
    for name, model, X in cases:
        with B.Forest(model) as f:
            ran = []
            for k in KERNELS:
                if supported(f, k):
                    print(f"[max] {name} {B.KERNEL_NAMES[k]}", flush=True)
                    check_parity(model, X, k, f"{name} {B.KERNEL_NAMES[k]}", forest=f)
                    ran.append(k)
            assert B.BRIDGER_KERNEL_DIRECT in ran
            if name == "perfect depth 10":
                assert B.BRIDGER_KERNEL_PERFECT in ran
            if name == "perfect depth 11":
                assert B.BRIDGER_KERNEL_PERFECT not in ran


def test_rows_beyond_one_launch():
    """More rows than one dispatch takes (2^24): the rows go out as several launches, so the
    rows on both sides of each launch boundary, CSR rows (whose entry offsets stay absolute),
    the Normalizer's per-launch norms and the binning pass must all line up."""
    import torch
    from oracle import binning
    from oracle import preprocess as P
    rng = np.random.default_rng(24)
    n = (1 << 24) + 4099
    X = rng.standard_normal((n, 2)).astype(np.float32)
    trees = [perfect_tree_arrays(2, rng.integers(0, 2, 3), rng.standard_normal(3).astype(np.float32) * 0.5,
                                 rng.standard_normal(4).astype(np.float32)) for _ in range(3)]
    model = concat_trees(trees, 2)
    ref, ref_lv = oracle_predict(model, X, leaves=True)
    Xd = to_dev(X)
    with B.Forest(model) as f:
        for k in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT):
            f.kernel = k
            what = f"{n} rows {B.KERNEL_NAMES[k]}"
            print(f"[big] {what}", flush=True)
            assert_scores(gpu_predict(f, Xd), ref, what)
            assert_leaves(gpu_predict(f, Xd, leaves=True), ref_lv, what)
        f.kernel = B.BRIDGER_KERNEL_PERFECT
        ip = torch.arange(0, 2 * n + 1, 2, dtype=torch.int64, device="cuda")
        ix = torch.tensor([0, 1], dtype=torch.int32, device="cuda").repeat(n)
        out = f.predict_csr(ip, ix, Xd.view(-1), n)
        torch.cuda.synchronize()
        assert_scores(out.cpu().numpy(), ref, "csr rows")
        del ip, ix, out
        q = f.bin(Xd)
        torch.cuda.synchronize()
        got = q.cpu().numpy().view(np.uint8 if f.bin_info()["bin_bytes"] == 1 else np.uint16)
        assert np.array_equal(got.astype(np.int64), binning.bin_rows(binning.tables(model), X)), "bins"
        f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)
        refn, _ = oracle_predict(model, P.apply(P.NORMALIZE, None, None, X))
        assert_scores(gpu_predict(f, Xd), refn, "normalized rows")
