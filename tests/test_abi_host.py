"""Host-side checks that need no GPU: the library loads and exports every declared entry
point; create validates forests; the packed layouts, walked by a test-only interpreter on
the CPU, reproduce the oracle; the launch plan respects the LDS capacity."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2405_12491_amd as B
from synth import (AGG_MEAN, XFORM_SIGMOID, XFORM_SOFTMAX, CONFIGS, concat_trees, make_workload,
                   perfect_tree_arrays, permute_nodes, random_tiny_forest)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bridger.h")


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bridger_\w+)\s*\(", text)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("bridger_forest_create", "bridger_forest_predict", "bridger_forest_predict_leaves",
              "bridger_forest_destroy", "bridger_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_calibration_library_exports_its_symbols():
    """include/bridger_calib.h is implemented by libbridger_calib.so; every header under
    include/ is covered by one of the two libraries."""
    headers = sorted(os.listdir(os.path.join(ROOT, "include")))
    assert headers == ["bridger.h", "bridger_calib.h"]
    lib = ctypes.CDLL(os.path.join(os.path.dirname(B.LIB_PATH), "libbridger_calib.so"))
    names = declared_functions(os.path.join(ROOT, "include", "bridger_calib.h"))
    assert set(names) == {"bridger_calib_device", "bridger_calib_lds_gather",
                          "bridger_calib_global_gather", "bridger_calib_copy"}
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def host(model, **kw):
    return B.Forest(model, host_only=True, **kw)


def _tiny():
    return concat_trees([perfect_tree_arrays(2, np.array([0, 1, 1]), np.array([0.5, 0.25, 0.75], np.float32),
                                             np.array([1, 2, 3, 4], np.float32))], 2)


def _create_err(**changes):
    f = _tiny()
    args = dict(n_trees=f.n_trees, tree_offsets=f.tree_offsets, feature=f.feature, threshold=f.threshold,
                left=f.left, right=f.right, value=f.value, n_features=2, n_classes=1, tree_class=None,
                aggregate=0, transform=0, base_score=None, flags=B.BRIDGER_CREATE_HOST_ONLY)
    args.update(changes)
    with pytest.raises(B.BridgerError) as e:
        B.bridger_forest_create(**args)
    return e.value.status


def test_validation_errors():
    f = _tiny()
    INV, ARG, UNS = B.BRIDGER_ERR_INVALID_FOREST, B.BRIDGER_ERR_INVALID_ARGUMENT, B.BRIDGER_ERR_UNSUPPORTED
    l = f.left.copy(); l[1] = 0                                   # root as a child (cycle)
    assert _create_err(left=l) == INV
    l = f.left.copy(); l[2] = 9                                   # child out of range
    assert _create_err(left=l) == INV
    l = f.left.copy(); l[1] = -1                                  # exactly one child
    assert _create_err(left=l) == INV
    l = f.left.copy(); r = f.right.copy(); l[0] = 1; r[0] = 1     # identical children
    assert _create_err(left=l, right=r) == INV
    l = f.left.copy(); l[1] = 4                                   # node 4 has two parents, 3 unreachable
    assert _create_err(left=l) == INV
    ft = f.feature.copy(); ft[0] = 2                              # feature >= n_features
    assert _create_err(feature=ft) == INV
    ft = f.feature.copy(); ft[0] = -3
    assert _create_err(feature=ft) == INV
    th = f.threshold.copy(); th[1] = np.nan                       # NaN threshold
    assert _create_err(threshold=th) == INV
    assert _create_err(n_trees=0, tree_offsets=np.zeros(1, np.int64)) == ARG
    assert _create_err(tree_offsets=np.array([1, 7], np.int64)) == INV
    assert _create_err(n_features=0) == ARG
    assert _create_err(n_classes=0) == ARG
    assert _create_err(n_classes=65) == UNS
    assert _create_err(transform=XFORM_SIGMOID, n_classes=2) == ARG
    assert _create_err(transform=XFORM_SOFTMAX) == ARG
    assert _create_err(tree_class=np.array([3], np.int32), n_classes=2) == ARG
    assert _create_err(aggregate=AGG_MEAN, n_classes=2, tree_class=np.array([1], np.int32)) == ARG
    assert _create_err(aggregate=7) == ARG
    assert _create_err(flags=8) == ARG
    # vector leaves: [N, K] values, no tree_class
    f = _tiny()
    v2 = np.stack([f.value, 1 - f.value], 1)
    assert _create_err(value=v2, n_classes=2, tree_class=np.array([1], np.int32)) == ARG


def test_vector_leaf_forest_on_host():
    f = _tiny()
    for K in (1, 3):
        v = np.repeat(f.value[:, None], K, 1) * np.arange(1, K + 1, dtype=np.float32)[None, :]
        h = B.bridger_forest_create(f.n_trees, f.tree_offsets, f.feature, f.threshold, f.left,
                                    f.right, v, 2, K, None, AGG_MEAN, 0, None,
                                    B.BRIDGER_CREATE_HOST_ONLY)
        info = B.bridger_forest_info(h)
        assert info["n_outputs"] == K and info["all_perfect"] == 1
        B.load_library().bridger_forest_destroy(h)


def test_vector_leaf_rows_in_perfect_blocks():
    """Vector leaves of at most 4 classes: each perfect tree block holds its leaves' class rows
    (16 bytes, zero-padded) in place of the scalar values, 24 * 2^D bytes per tree, so that the
    tree chunks bring them to LDS; more classes keep the 12 * 2^D block."""
    rng = np.random.default_rng(5)
    D, T, n_leaf = 3, 3, 8
    trees = [perfect_tree_arrays(D, rng.integers(0, 4, 7), rng.standard_normal(7).astype(np.float32),
                                 rng.standard_normal(8).astype(np.float32)) for _ in range(T)]
    base = concat_trees(trees, 4)
    for K in (2, 3, 4, 5):
        v = rng.standard_normal((base.value.size, K)).astype(np.float32)
        h = B.bridger_forest_create(base.n_trees, base.tree_offsets, base.feature, base.threshold,
                                    base.left, base.right, v, 4, K, None, AGG_MEAN, 0, None,
                                    B.BRIDGER_CREATE_HOST_ONLY)
        try:
            blob = B.bridger_forest_packed(h, 0, np.uint8)
            leaf_map = B.bridger_forest_packed(h, 2, np.int32)
            order = B.bridger_forest_packed(h, 3, np.int32)
            tb = blob.size // T
            if K > 4:
                assert tb == 12 << D
                continue
            assert tb == 24 << D
            for k in range(T):
                rows = blob[k * tb + 8 * n_leaf:(k + 1) * tb].view(np.float32).reshape(n_leaf, 4)
                for j in range(n_leaf):
                    node = base.tree_offsets[order[k]] + leaf_map[k * n_leaf + j]
                    np.testing.assert_array_equal(rows[j, :K], v[node])
                    assert not rows[j, K:].any()
        finally:
            B.load_library().bridger_forest_destroy(h)


def test_null_pointer_arguments():
    lib = B.load_library()
    h = ctypes.c_void_p()
    st = lib.bridger_forest_create_ex(1, None, None, None, None, None, None, 2, 1, None, 0, 0, None,
                                      1, ctypes.byref(h))
    assert st == B.BRIDGER_ERR_INVALID_ARGUMENT and not h.value
    assert lib.bridger_forest_predict(None, None, 1, 2, None, None) == B.BRIDGER_ERR_INVALID_ARGUMENT
    assert "null" in B.bridger_last_error()
    lib.bridger_forest_destroy(None)


def test_deep_tree_rejected():
    # a chain of depth 65
    n = 131
    left = np.full(n, -1, np.int32); right = np.full(n, -1, np.int32)
    for d in range(65):
        left[2 * d] = 2 * d + 1 if 2 * d + 1 < n else -1
        right[2 * d] = 2 * d + 2
    f = concat_trees([(np.zeros(n, np.int32), np.zeros(n, np.float32), left, right, np.zeros(n, np.float32))], 1)
    with pytest.raises(B.BridgerError) as e:
        host(f)
    assert e.value.status == B.BRIDGER_ERR_INVALID_FOREST


def test_predict_on_host_only_handle_fails():
    with host(_tiny()) as f:
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_predict(f.handle, 16, 1, 2, 64, 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT


def test_noalloc_size_limit():
    """The allocation-free predict rejects more rows than its scratch holds, before anything
    else is checked (so on a host-only handle too); the header and binding agree on the limit."""
    text = open(HEADER).read()
    m = re.search(r"#define BRIDGER_NOALLOC_MAX_ROWS (\d+)", text)
    assert m and int(m.group(1)) == B.NOALLOC_MAX_ROWS
    with host(_tiny()) as f:
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_predict_noalloc(f.handle, 16, B.NOALLOC_MAX_ROWS + 1, 2, 64, 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        assert "allocation-free limit" in B.bridger_last_error()
        with pytest.raises(B.BridgerError) as e:   # within the limit: the host-only handle
            B.bridger_forest_predict_noalloc(f.handle, 16, 1, 2, 64, 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        assert "host-only" in B.bridger_last_error()


# ----------------------------------------------------- packed-layout interpreter
def walk_perfect(f: B.Forest, model, X):
    """1-based heap: slot m at byte 8m (children 2m, 2m+1), leaves from byte 8*2^D."""
    blob = B.bridger_forest_packed(f.handle, 0, np.uint8)
    leaf_map = B.bridger_forest_packed(f.handle, 2, np.int32)
    order = B.bridger_forest_packed(f.handle, 3, np.int32)
    D = f.info()["max_depth"]
    T = f.n_trees
    tb = blob.size // T
    assert tb == 12 << D
    n_leaf = 1 << D
    leaves = np.empty((X.shape[0], T), np.int32)
    vals = np.empty((X.shape[0], T), np.float32)
    rows = np.arange(X.shape[0])
    for k in range(T):
        blk = blob[k * tb:(k + 1) * tb]
        thr = blk[:8 * n_leaf].view(np.float32)[0::2]
        feat = blk[:8 * n_leaf].view(np.uint32)[1::2]
        lv = blk[8 * n_leaf:12 * n_leaf].view(np.float32)
        m = np.ones(X.shape[0], np.int64)
        for _ in range(D):
            m = 2 * m + np.where(X[rows, feat[m]] <= thr[m], 0, 1)
        j = m - n_leaf
        leaves[:, order[k]] = leaf_map[k * n_leaf + j]
        vals[:, order[k]] = lv[j]
    return leaves, vals


def walk_ragged(f: B.Forest, X):
    rec = B.bridger_forest_packed(f.handle, 0, np.uint32).reshape(-1, 2)
    start = B.bridger_forest_packed(f.handle, 1, np.int32)
    rec_node = B.bridger_forest_packed(f.handle, 2, np.int32)
    order = B.bridger_forest_packed(f.handle, 3, np.int32)
    T = f.n_trees
    leaves = np.empty((X.shape[0], T), np.int32)
    vals = np.empty((X.shape[0], T), np.float32)
    rows = np.arange(X.shape[0])
    for k in range(T):
        a = np.full(X.shape[0], start[k], np.int64)
        for _ in range(70):
            meta = rec[a, 1]
            leaf = (meta & 0x8000) != 0
            if leaf.all():
                break
            feat = (meta >> 16).astype(np.int64)
            right = ~(X[rows, feat] <= rec[a, 0].view(np.float32)) & ~leaf
            a = np.where(leaf, a, a + (meta & 0x7FFF) + right)
        assert np.all((rec[a, 1] & 0x8000) != 0)
        nxt = a + (rec[a, 1] & 0x7FFF)
        assert np.all(nxt == start[k + 1])                     # a leaf points at the next root
        leaves[:, order[k]] = rec_node[a]
        vals[:, order[k]] = rec[a, 0].view(np.float32)
    return leaves, vals


def has_tops(f: B.Forest) -> bool:
    try:
        B.bridger_forest_packed(f.handle, 7, np.uint32)
        return True
    except B.BridgerError:
        return False


def walk_ragged_tops(f: B.Forest, X):
    """The lockstep kernel's walk: levels 0-3 from the top-level heaps (slot 0 the root's record
    index, slot m's children at 2m and 2m + 1), deeper levels from the packed records.  Every
    heap record must equal the packed record at the index the walk tracks."""
    rec = B.bridger_forest_packed(f.handle, 0, np.uint32).reshape(-1, 2)
    tops = B.bridger_forest_packed(f.handle, 7, np.uint32).reshape(-1, 2)
    rec_node = B.bridger_forest_packed(f.handle, 2, np.int32)
    order = B.bridger_forest_packed(f.handle, 3, np.int32)
    T = f.n_trees
    # L top levels: 2^L records per tree, then 1024 / (8 * 2^L) empty trees
    L = [l for l in (4, 5) if tops.shape[0] == (T + 1024 // (8 << l)) << l]
    assert len(L) == 1
    L = L[0]
    tops = tops.reshape(-1, 1 << L, 2)
    assert np.all(tops[T:, 1:, 1] == 0x8000)
    leaves = np.empty((X.shape[0], T), np.int32)
    rows = np.arange(X.shape[0])
    for k in range(T):
        a = np.full(X.shape[0], tops[k, 0, 0], np.int64)
        m = np.ones(X.shape[0], np.int64)
        r = tops[k, 1][None, :].repeat(X.shape[0], 0)
        for level in range(70):
            assert np.array_equal(r, rec[a])
            meta = r[:, 1]
            leaf = (meta & 0x8000) != 0
            if leaf.all():
                break
            feat = (meta >> 16).astype(np.int64)
            right = (~(X[rows, feat] <= r[:, 0].view(np.float32)) & ~leaf).astype(np.int64)
            a = np.where(leaf, a, a + (meta & 0x7FFF) + right)
            m = np.where(leaf, m, 2 * m + right)
            r = tops[k][m] if level + 1 < L else rec[a]
        leaves[:, order[k]] = rec_node[a]
    return leaves


def walk_direct(f: B.Forest, X):
    rec = B.bridger_forest_packed(f.handle, 0, np.int32).reshape(-1, 4)
    root = B.bridger_forest_packed(f.handle, 1, np.int32)
    rec_node = B.bridger_forest_packed(f.handle, 2, np.int32)
    order = B.bridger_forest_packed(f.handle, 3, np.int32)
    T = f.n_trees
    leaves = np.empty((X.shape[0], T), np.int32)
    rows = np.arange(X.shape[0])
    for k in range(T):
        n = np.full(X.shape[0], root[k], np.int64)
        while True:
            feat = rec[n, 1]
            act = feat >= 0
            if not act.any():
                break
            go_left = X[rows, np.maximum(feat, 0)] <= rec[n, 0].view(np.float32)
            n = np.where(act, np.where(go_left, rec[n, 2], rec[n, 3]), n)
        leaves[:, order[k]] = rec_node[n]
    return leaves


@pytest.mark.parametrize("name", list(CONFIGS))
def test_packed_layouts_reproduce_oracle_leaves(name):
    w = make_workload(name, 200 if name != "ragged_d12" else 40)
    X = w.X()
    _, ref_lv, _ = oracle.predict(w.forest, X, want_leaves=True, threads=8)
    with host(w.forest) as f:
        for k in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT):
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            if k == B.BRIDGER_KERNEL_PERFECT:
                lv, _ = walk_perfect(f, w.forest, X)
            elif k == B.BRIDGER_KERNEL_RAGGED:
                lv, _ = walk_ragged(f, X)
                if has_tops(f):
                    assert np.array_equal(walk_ragged_tops(f, X), ref_lv), name
            else:
                lv = walk_direct(f, X)
            assert np.array_equal(lv, ref_lv), (name, k)


@pytest.mark.parametrize("levels", ["4", "5"])
@pytest.mark.parametrize("seed", range(6))
def test_ragged_top_heaps(seed, levels, monkeypatch):
    """Random ragged one-class forests (leaves at every top level, single-leaf trees, trees
    shallower than the heap) get top-level heaps, and walking them reproduces the oracle."""
    monkeypatch.setenv("BRIDGER_TOP_LEVELS", levels)
    rng = np.random.default_rng(100 + seed)
    F = int(rng.integers(1, 9))
    model = random_tiny_forest(rng, int(rng.integers(1, 40)), F, max_depth=int(rng.integers(0, 9)),
                               p_split=float(rng.uniform(0.3, 0.95)), thr_grid=[-1.0, 0.0, 0.5, 1.0])
    model = permute_nodes(model, rng)
    X = rng.choice(np.array([-1.0, 0.0, 0.5, 1.0, 2.0, np.nan], np.float32), (64, F))
    _, ref_lv, _ = oracle.predict(model, X, want_leaves=True)
    with host(model) as f:
        if f.kernel != B.BRIDGER_KERNEL_RAGGED:
            f.kernel = B.BRIDGER_KERNEL_RAGGED
        assert has_tops(f)
        assert np.array_equal(walk_ragged_tops(f, X), ref_lv)


def test_packed_layouts_permuted_and_classes():
    rng = np.random.default_rng(5)
    trees = [perfect_tree_arrays(3, rng.integers(0, 5, 7), rng.standard_normal(7).astype(np.float32),
                                 rng.standard_normal(8).astype(np.float32)) for _ in range(11)]
    model = permute_nodes(concat_trees(trees, 5, 3, rng.integers(0, 3, 11)), rng)
    X = rng.standard_normal((300, 5)).astype(np.float32)
    _, ref_lv, _ = oracle.predict(model, X, want_leaves=True)
    with host(model) as f:
        order = B.bridger_forest_packed(f.handle, 3, np.int32)
        tc = model.tree_class[order]
        assert np.all(np.diff(tc) >= 0)                            # class-major
        for c in range(3):                                         # stable within a class
            assert np.all(np.diff(order[tc == c]) > 0)
        lv, _ = walk_perfect(f, model, X)
        assert np.array_equal(lv, ref_lv)
        f.kernel = B.BRIDGER_KERNEL_RAGGED
        lv, _ = walk_ragged(f, X)
        assert np.array_equal(lv, ref_lv)
    rf = random_tiny_forest(rng, 17, 4, max_depth=8)
    X = rng.standard_normal((300, 4)).astype(np.float32)
    _, ref_lv, _ = oracle.predict(rf, X, want_leaves=True)
    with host(rf) as f:
        assert f.kernel == B.BRIDGER_KERNEL_RAGGED
        lv, _ = walk_ragged(f, X)
        assert np.array_equal(lv, ref_lv)


@pytest.mark.parametrize("K", [1, 3, 8, 10])
def test_class_sums_share_the_row_tile(K):
    """Chunked PERFECT plans for at most 8 classes keep the class sums in registers and write
    them into the row tile after the walk: the LDS is the tile plus two chunk buffers.  More
    classes reserve K x G x R doubles of class slots on top."""
    import dataclasses
    w = make_workload("gbdt_d6", 1000)
    model = w.forest if K == 1 else dataclasses.replace(
        w.forest, n_classes=K, tree_class=(np.arange(w.forest.n_trees) % K).astype(np.int32),
        transform=XFORM_SOFTMAX, base_score=np.zeros(K, np.float32))
    with host(model) as f:
        p = f.plan(1_000_000)
        R, F = p["rows_per_wg"], w.n_features
        assert p["chunk_bytes"] > 0
        tile_and_chunks = 2 * p["chunk_bytes"] + R * F * 4
        if K <= 8:
            assert p["lds_bytes"] == tile_and_chunks
        else:
            assert p["lds_bytes"] >= tile_and_chunks + 8 * K * R


@pytest.mark.parametrize("name", list(CONFIGS))
def test_plan_respects_lds_capacity(name):
    w = make_workload(name, 1000)
    with host(w.forest) as f:
        for k in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            p = f.plan(w.n_rows)
            R = p["rows_per_wg"]
            assert R >= 32 and R & (R - 1) == 0
            assert p["lds_bytes"] <= 160 * 1024
            assert 2 * p["chunk_bytes"] + R * w.n_features * 4 <= p["lds_bytes"]
            if k == B.BRIDGER_KERNEL_PERFECT and p["chunk_bytes"] == 0:
                # records read from global memory: the LDS holds the tile and class sums only
                assert p["trees_per_chunk"] == 0 and p["n_chunks"] == 0
                assert R * w.n_features * 4 + 8 * f.n_classes * R <= p["lds_bytes"]
            elif k == B.BRIDGER_KERNEL_PERFECT:
                tb = B.bridger_forest_packed(f.handle, 0, np.uint8).size // f.n_trees
                assert p["trees_per_chunk"] * tb <= p["chunk_bytes"]
                assert p["n_chunks"] * p["trees_per_chunk"] >= f.n_trees
            elif p["chunk_bytes"] == 0:
                # records read from global memory: no chunks
                assert p["n_chunks"] == 0
                assert R * w.n_features * 4 <= p["lds_bytes"]
            else:
                chunks = B.bridger_forest_packed(f.handle, 4, np.int32)
                start = B.bridger_forest_packed(f.handle, 1, np.int32)
                assert chunks[0] == 0 and chunks[-1] == f.n_trees
                assert len(chunks) - 1 == p["n_chunks"]
                for a, b in zip(chunks[:-1], chunks[1:]):
                    assert 8 * (start[b] - start[a]) <= p["chunk_bytes"]
                    assert start[a] % 2 == 0                    # 16-byte aligned chunk start


def test_create_without_gpu_reports_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(B.BridgerError) as e:
        B.Forest(_tiny())
    assert e.value.status == B.BRIDGER_ERR_DEVICE


def _deep_tree_bytes(D, TL):
    pairs = sum(16 << (TL + 2 * j) for j in range((D - TL) // 2))
    return pairs + ((16 << (D - 1)) if (D - TL) & 1 else (4 << D))


def walk_perfect_deep(f: B.Forest, X, D, TL, bins=None):
    """The wide-row perfect walk: the first TL levels from the packed records (the LDS copies
    hold the same records), then the deep blocks (packed array 8; with bins, array 9, whose
    w fields are ranks and a row goes right iff its bin exceeds the rank)."""
    blob = B.bridger_forest_packed(f.handle, 0, np.uint8)
    deep = B.bridger_forest_packed(f.handle, 9 if bins is not None else 8, np.uint8)
    leaf_map = B.bridger_forest_packed(f.handle, 2, np.int32)
    order = B.bridger_forest_packed(f.handle, 3, np.int32)
    T = f.n_trees
    tb, dtb = blob.size // T, deep.size // T
    assert dtb == _deep_tree_bytes(D, TL), (D, TL, dtb)
    n = X.shape[0]
    rows = np.arange(n)
    leaves = np.empty((n, T), np.int32)
    vals = np.empty((n, T), np.float32)

    def right(w, x_or_bin):
        if bins is not None:
            return (x_or_bin > w.astype(np.int64)).astype(np.int64)
        return np.where(x_or_bin <= w.view(np.float32), 0, 1)

    V = bins if bins is not None else X
    for k in range(T):
        blk = blob[k * tb:(k + 1) * tb]
        thr = blk[:8 << D].view(np.float32)[0::2]
        feat = blk[:8 << D].view(np.uint32)[1::2]
        m = np.ones(n, np.int64)
        for _ in range(TL):   # top levels: fp32 thresholds of the records (bins: ranks below)
            if bins is None:
                m = 2 * m + np.where(X[rows, feat[m]] <= thr[m], 0, 1)
            else:
                ranks = {i: _rank(f, int(feat[i]), thr[i]) for i in np.unique(m)}
                w = np.array([ranks[i] for i in m], np.uint32)
                m = 2 * m + right(w, bins[rows, feat[m]])
        d_blk = deep[k * dtb:(k + 1) * dtb].view(np.uint32)
        off = 0
        d = TL
        while D - d >= 2:
            q = d_blk[off // 4:off // 4 + (4 << d)].reshape(-1, 4)[m - (1 << d)]
            b1 = right(q[:, 0].copy(), V[rows, q[:, 3] & 1023])
            w2 = np.where(b1 == 1, q[:, 2], q[:, 1]).astype(np.uint32)
            f2 = (q[:, 3] >> np.where(b1 == 1, 20, 10).astype(np.uint32)) & 1023
            b2 = right(w2, V[rows, f2])
            m = 4 * m + 2 * b1 + b2
            off += 16 << d
            d += 2
        if d == D - 1:
            q = d_blk[off // 4:off // 4 + (4 << d)].reshape(-1, 4)[m - (1 << d)]
            b = right(q[:, 0].copy(), V[rows, q[:, 1]])
            lv = np.where(b == 1, q[:, 3], q[:, 2]).view(np.float32)
            m = 2 * m + b
        else:
            assert d == D
            lv = d_blk[off // 4:off // 4 + (1 << D)].view(np.float32)[m - (1 << D)]
        leaves[:, order[k]] = leaf_map[k * (1 << D) + m - (1 << D)]
        vals[:, order[k]] = lv
    return leaves, vals


def _rank(f: B.Forest, feat: int, t: float) -> int:
    """A threshold's rank among its feature's binning thresholds (packed arrays 5 and 6)."""
    q = B.bridger_forest_packed(f.handle, 5, np.float32)
    qo = B.bridger_forest_packed(f.handle, 6, np.int32)
    u = q[qo[feat]:qo[feat + 1]]
    return int(np.searchsorted(u, np.float32(t) + np.float32(0.0), side="left"))


@pytest.mark.parametrize("D,F,levels", [(4, 7, "3"), (5, 9, "3"), (6, 28, "3"), (7, 5, "3"),
                                        (8, 784, "3"), (8, 1024, "4"), (9, 12, "4"), (10, 3, "3")])
def test_perfect_deep_blocks(D, F, levels, monkeypatch):
    """The deep blocks of the wide-row perfect kernel (pairs of levels in one 16-byte block,
    the last level with its leaf values, or a leaf array) walked on the CPU reach the oracle's
    leaves and values: fp32 rows with ties, signed zeros, infinities and NaN, and bins."""
    monkeypatch.setenv("BRIDGER_PERFECT_TOP_LEVELS", levels)
    rng = np.random.default_rng(D * 100 + F)
    T = 9
    n_int = (1 << D) - 1
    grid = np.array([-1.0, -0.0, 0.0, 0.5, 1.0, np.inf], np.float32)
    trees = [perfect_tree_arrays(D, rng.integers(0, F, n_int),
                                 rng.choice(grid, n_int).astype(np.float32),
                                 rng.standard_normal(1 << D).astype(np.float32))
             for _ in range(T)]
    model = permute_nodes(concat_trees(trees, F), rng)
    X = rng.choice(np.array([-2.0, -1.0, -0.0, 0.0, 0.5, 1.0, 3.0, np.inf, -np.inf, np.nan],
                            np.float32), (200, F))
    _, ref_lv, _ = oracle.predict(model, X, want_leaves=True)
    ref_val = model.value[model.tree_offsets[:-1][None, :] + ref_lv]
    with host(model) as f:
        assert f.kernel == B.BRIDGER_KERNEL_PERFECT
        lv, vals = walk_perfect_deep(f, X, D, int(levels))
        assert np.array_equal(lv, ref_lv)
        assert np.array_equal(vals, ref_val.astype(np.float32))
        from oracle import binning
        bins = binning.bin_rows(binning.tables(model), X)
        lv, vals = walk_perfect_deep(f, X, D, int(levels), bins=bins)
        assert np.array_equal(lv, ref_lv)
        assert np.array_equal(vals, ref_val.astype(np.float32))


def test_perfect_deep_blocks_absent():
    """More than 1024 features or vector leaves: no deep blocks (the kernel reads every level
    from the records)."""
    rng = np.random.default_rng(3)
    trees = [perfect_tree_arrays(6, rng.integers(0, 1100, 63), rng.standard_normal(63).astype(np.float32),
                                 rng.standard_normal(64).astype(np.float32)) for _ in range(3)]
    with host(concat_trees(trees, 1100)) as f:
        with pytest.raises(B.BridgerError):
            B.bridger_forest_packed(f.handle, 8, np.uint8)


def walk_treelets(f: B.Forest, X, bins=None):
    """The treelet walk (packed arrays 10-12; with bins, 13 and right iff bin > rank): slot s of
    a tree holds a node and its two children; a leaf child ends the walk, an internal one moves
    it to slot 4s + 1 + 2 b1 + b2."""
    blk = B.bridger_forest_packed(f.handle, 13 if bins is not None else 10, np.uint32).reshape(-1, 4)
    start = B.bridger_forest_packed(f.handle, 11, np.int32)
    leaf_ids = B.bridger_forest_packed(f.handle, 12, np.int32)
    order = B.bridger_forest_packed(f.handle, 3, np.int32)
    T = f.n_trees
    n = X.shape[0]
    rows = np.arange(n)
    V = bins if bins is not None else X

    def right(w, x):
        if bins is not None:
            return (x > w.astype(np.int64)).astype(np.int64)
        return np.where(x <= w.view(np.float32), 0, 1)

    leaves = np.empty((n, T), np.int32)
    vals = np.empty((n, T), np.float32)
    for k in range(T):
        s = np.zeros(n, np.int64)
        done = np.zeros(n, bool)
        lid = np.zeros(n, np.int64)
        val = np.zeros(n, np.uint32)
        for _ in range(40):
            if done.all():
                break
            q = blk[start[k] + s]
            b1 = right(q[:, 0].copy(), V[rows, q[:, 3] & 1023])
            wc = np.where(b1 == 1, q[:, 2], q[:, 1]).astype(np.uint32)
            fc = (q[:, 3] >> np.where(b1 == 1, 20, 10).astype(np.uint32)) & 1023
            leaf = ((q[:, 3] >> (30 + b1).astype(np.uint32)) & 1) == 1
            fin = ~done & leaf
            lid[fin] = (start[k] + s[fin]) * 2 + b1[fin]
            val[fin] = wc[fin]
            go = ~done & ~leaf
            b2 = right(wc, V[rows, fc])
            s = np.where(go, 4 * s + 1 + 2 * b1 + b2, s)
            done |= fin
        assert done.all()
        leaves[:, order[k]] = leaf_ids[lid]
        vals[:, order[k]] = val.view(np.float32)
    return leaves, vals


@pytest.mark.parametrize("seed", range(6))
def test_ragged_treelets(seed):
    """Random one-class ragged forests (single-leaf trees, leaves at every level, depths up to
    11, ties, NaN and infinite inputs) packed as two-level treelets: walking them reproduces
    the oracle's leaf ids and leaf values, on fp32 rows and on bins."""
    rng = np.random.default_rng(300 + seed)
    F = int(rng.integers(1, 12))
    model = random_tiny_forest(rng, int(rng.integers(1, 30)), F, max_depth=int(rng.integers(0, 12)),
                               p_split=float(rng.uniform(0.3, 0.95)), thr_grid=[-1.0, -0.0, 0.0, 0.5, 1.0])
    model = permute_nodes(model, rng)
    X = rng.choice(np.array([-1.0, -0.0, 0.0, 0.5, 1.0, 2.0, np.nan, np.inf, -np.inf], np.float32), (96, F))
    _, ref_lv, _ = oracle.predict(model, X, want_leaves=True)
    ref_val = model.value[model.tree_offsets[:-1][None, :] + ref_lv].astype(np.float32)
    with host(model) as f:
        if f.kernel != B.BRIDGER_KERNEL_RAGGED:
            f.kernel = B.BRIDGER_KERNEL_RAGGED
        if not has_tops(f):
            pytest.skip("plan without top levels")
        lv, vals = walk_treelets(f, X)
        assert np.array_equal(lv, ref_lv)
        assert np.array_equal(vals, ref_val)
        from oracle import binning
        bins = binning.bin_rows(binning.tables(model), X)
        lv, vals = walk_treelets(f, X, bins=bins)
        assert np.array_equal(lv, ref_lv)
        assert np.array_equal(vals, ref_val)
