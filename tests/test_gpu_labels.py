"""GPU parity of classifier labels: argmax of the class values (several classes) or the sign
of the margin (one sigmoid output), against labels taken from the oracle's outputs.  Where
the oracle's top two values lie within rounding distance, either label is accepted."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import check_labels as _check_labels, oracle_predict, to_dev
from synth import (AGG_MEAN, XFORM_IDENTITY, XFORM_SOFTMAX, make_workload, random_tiny_forest)

pytestmark = pytest.mark.gpu

KERNELS = [B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED, B.BRIDGER_KERNEL_DIRECT,
           B.BRIDGER_KERNEL_GEMM]


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


@pytest.mark.parametrize("case", ["mc_gbdt_d8", "gbdt_d6", "shallow_d3", "ragged_mean3",
                                  "ragged_mean3_chunked"])
def test_labels(case, monkeypatch):
    import torch
    if case.endswith("_chunked"):   # ragged trees through LDS chunks instead of global records
        monkeypatch.setenv("BRIDGER_GLOBAL", "0")
        case = case[:-len("_chunked")]
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
