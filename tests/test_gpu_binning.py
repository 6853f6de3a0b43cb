"""GPU parity of exact feature quantization: the binning kernel against the binning oracle
(bit-exact), and prediction on bins against the fp32 oracle (scores within tolerance, leaf
ids bit-exact), through the C ABI."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from oracle import binning
from parity_util import assert_leaves, assert_scores, oracle_predict, to_dev
from synth import (AGG_MEAN, CONFIGS, EXTRA_CONFIGS, XFORM_SOFTMAX, concat_trees, make_workload,
                   perfect_tree_arrays, random_tiny_forest)
from test_binning import GRID, _adversarial_X

pytestmark = pytest.mark.gpu

SMALL_ROWS = {"dt_d3": 10_000, "rf_d8": 3 * 1024 + 77, "gbdt_d6": 3 * 1024 + 77,
              "mc_gbdt_d8": 2 * 32 * 3 + 45, "ragged_d12": 3 * 64 + 29,
              "shallow_d3": 2 * 1024 + 5, "shallow_d4": 2 * 1024 + 5,
              "ragged_rf_28": 2 * 512 + 37}


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _check_binned(model, X, what, kernel=None):
    import torch
    tabs = binning.tables(model)
    ref_bins = binning.bin_rows(tabs, X)
    ref, ref_lv = oracle_predict(model, X, leaves=True)
    with B.Forest(model) as f:
        if kernel is not None:
            f.kernel = kernel
        Xd = to_dev(X)
        q = f.bin(Xd)
        torch.cuda.synchronize()
        bb = f.bin_info()["bin_bytes"]
        got_bins = q.cpu().numpy().view(np.uint8 if bb == 1 else np.uint16).astype(np.int64)
        assert np.array_equal(got_bins, ref_bins), f"{what}: bins differ from the oracle"
        out = f.predict_binned(q)
        lv = f.predict_binned_leaves(q)
        torch.cuda.synchronize()
        assert_scores(out.cpu().numpy().astype(np.float64), ref, what + " binned scores")
        assert_leaves(lv.cpu().numpy(), ref_lv, what + " binned leaves")
        return bb, B.KERNEL_NAMES[f.kernel]


@pytest.mark.parametrize("name", list(CONFIGS) + list(EXTRA_CONFIGS))
def test_binned_workloads(name):
    w = make_workload(name, SMALL_ROWS[name])
    X = w.X()
    for k in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
        with B.Forest(w.forest, host_only=True) as h:
            try:
                h.kernel = k
            except B.BridgerError:
                continue
        print(f"[binned] {name} rows={X.shape[0]} kernel={B.KERNEL_NAMES[k]}", flush=True)
        bb, kn = _check_binned(w.forest, X, f"{name}/{B.KERNEL_NAMES[k]}", kernel=k)
        print(f"[binned] {name} ok: {bb}-byte bins on {kn}", flush=True)


@pytest.mark.parametrize("F", [3, 7, 28])
def test_binned_adversarial(F):
    """NaN, +-inf, +-0, denormals, +-FLT_MAX and values one ulp around thresholds (8-bit bins)."""
    rng = np.random.default_rng(200 + F)
    G = len(GRID)
    perfect = concat_trees([perfect_tree_arrays(4, rng.integers(0, F, 15), GRID[rng.integers(0, G, 15)],
                                                rng.standard_normal(16).astype(np.float32))
                            for _ in range(9)], F)
    ragged = random_tiny_forest(rng, 15, F, max_depth=6, p_split=0.8, thr_grid=GRID)
    X = _adversarial_X(rng, binning.tables(perfect), F, n=700)
    for model, what in ((perfect, "perfect"), (ragged, "ragged")):
        bb, kn = _check_binned(model, X, f"adversarial F={F} {what}")
        assert bb == 1


@pytest.mark.parametrize("env", [{"BRIDGER_GLOBAL": "1"}, {"BRIDGER_GLOBAL": "0"},
                                 {"BRIDGER_GLOBAL": "1", "BRIDGER_DEEP": "0"},
                                 {"BRIDGER_TREELETS": "0"}, {"BRIDGER_TREELET_LDS_LEVELS": "2"},
                                 {"BRIDGER_GLOBAL": "1", "BRIDGER_PERFECT_TOP_LEVELS": "3"},
                                 {"BRIDGER_ILP": "1", "BRIDGER_WAVES": "4", "BRIDGER_ROWS": "128"},
                                 # the binning pass: row kernel, stream kernel, small LDS buffers
                                 # (many runs; tables larger than the buffer searched in place)
                                 {"BRIDGER_BIN_KERNEL": "1"}, {"BRIDGER_BIN_KERNEL": "2"},
                                 {"BRIDGER_BIN_KERNEL": "1", "BRIDGER_BIN_LDS_KB": "1"},
                                 {"BRIDGER_BIN_KERNEL": "1", "BRIDGER_BIN_CHUNKS": "3"},
                                 {"BRIDGER_BIN_KERNEL": "2", "BRIDGER_BIN_LDS_KB": "1"}],
                         ids=lambda e: ",".join(f"{k[8:]}={v}" for k, v in e.items()))
def test_binned_kernel_variants(env, monkeypatch):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    rng = np.random.default_rng(31)
    g = make_workload("gbdt_d6", 1500)
    multi = random_tiny_forest(rng, 40, 6, max_depth=8, n_classes=3, aggregate=AGG_MEAN,
                               transform=XFORM_SOFTMAX)
    X6 = rng.standard_normal((900, 6)).astype(np.float32)
    r = make_workload("ragged_d12", 200)
    for model, X, what in ((g.forest, g.X(), "gbdt_d6"), (multi, X6, "multiclass ragged"),
                           (r.forest, r.X(), "ragged_d12")):
        print(f"[binned] variant {env} {what}", flush=True)
        _check_binned(model, X, f"{what} {env}")


def test_binned_errors():
    import torch
    w = make_workload("gbdt_d6", 64)
    Xd = to_dev(w.X())
    with B.Forest(w.forest) as f:
        q = f.bin(Xd)
        out = torch.empty((64, 1), device="cuda")
        with pytest.raises(B.BridgerError) as e:   # Xq misaligned for 16-bit bins
            B.bridger_forest_predict_binned(f.handle, q.data_ptr() + 1, 64, 28, out.data_ptr(), 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        with pytest.raises(B.BridgerError) as e:   # wrong feature count
            B.bridger_forest_bin(f.handle, Xd.data_ptr(), 64, 27, q.data_ptr(), 0)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
        f.kernel = B.BRIDGER_KERNEL_DIRECT
        with pytest.raises(B.BridgerError) as e:   # binned rows need the perfect or ragged kernel
            f.predict_binned(q, out)
        assert e.value.status == B.BRIDGER_ERR_UNSUPPORTED
    n = 70_000
    t = np.arange(n, dtype=np.float32)
    model = concat_trees([perfect_tree_arrays(1, np.array([0]), t[i:i + 1], np.array([0.0, 1.0], np.float32))
                          for i in range(n)], 1)
    with B.Forest(model) as f:
        X1 = to_dev(np.zeros((8, 1), np.float32))
        q = torch.empty((8, 1), dtype=torch.int16, device="cuda")
        with pytest.raises(B.BridgerError) as e:
            B.bridger_forest_bin(f.handle, X1.data_ptr(), 8, 1, q.data_ptr(), 0)
        assert e.value.status == B.BRIDGER_ERR_UNSUPPORTED
