"""GPU parity of classifier labels: argmax of the class values (several classes) or the sign
of the margin (one sigmoid output), against labels taken from the oracle's outputs.  Where
the oracle's top two values lie within rounding distance, either label is accepted."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import oracle_predict, to_dev
from synth import (AGG_MEAN, XFORM_IDENTITY, XFORM_SOFTMAX, make_workload, random_tiny_forest)

pytestmark = pytest.mark.gpu

KERNELS = [B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT,
           B.BRIDGER_KERNEL_GEMM]
TIE = 1e-12


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _check_labels(got, ref, what):
    n, K = ref.shape
    if K == 1:
        want = (ref[:, 0] > 0.5).astype(np.int32)
        sure = np.abs(ref[:, 0] - 0.5) > TIE
    else:
        want = np.argmax(ref, axis=1).astype(np.int32)
        top = np.sort(ref, axis=1)
        sure = (top[:, -1] - top[:, -2]) > TIE * np.maximum(1.0, np.abs(top[:, -1]))
    bad = np.flatnonzero(sure & (got != want))
    assert bad.size == 0, f"{what}: {bad.size} labels differ, first row {bad[:1]}"
    for i in np.flatnonzero(~sure):   # near ties: any class within rounding of the top
        assert K > 1 and ref[i, got[i]] >= ref[i].max() - TIE * max(1.0, abs(ref[i].max())), what
    assert np.all((got >= 0) & (got < max(K, 2)))


@pytest.mark.parametrize("case", ["mc_gbdt_d8", "gbdt_d6", "shallow_d3", "ragged_mean3"])
def test_labels(case):
    import torch
    rng = np.random.default_rng(4)
    if case == "ragged_mean3":
        model = random_tiny_forest(rng, 30, 6, max_depth=8, n_classes=3, aggregate=AGG_MEAN,
                                   transform=XFORM_IDENTITY)
        X = rng.standard_normal((900, 6)).astype(np.float32)
    else:
        w = make_workload(case, {"mc_gbdt_d8": 300, "gbdt_d6": 2000, "shallow_d3": 1500}[case])
        model, X = w.forest, w.X()
    ref, _ = oracle_predict(model, X)
    Xd = to_dev(X)
    with B.Forest(model) as f:
        ran = 0
        for k in KERNELS:
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            got = f.predict_labels(Xd)
            torch.cuda.synchronize()
            _check_labels(got.cpu().numpy(), ref, f"{case} {B.KERNEL_NAMES[k]}")
            ran += 1
        assert ran >= 2


def test_labels_need_a_classifier():
    import torch
    w = make_workload("rf_d8", 64)   # one output, mean, no link: a regressor
    Xd = to_dev(w.X())
    with B.Forest(w.forest) as f:
        out = torch.empty(64, dtype=torch.int32, device="cuda")
        with pytest.raises(B.BridgerError) as e:
            f.predict_labels(Xd, out)
        assert e.value.status == B.BRIDGER_ERR_UNSUPPORTED
