"""Out-of-memory paths, forced from the host with the library's allocation-limit test hook
(BRIDGER_TEST_ALLOC_LIMIT: every device allocation larger than the limit fails as an exhausted
device would).  A refused create returns BRIDGER_ERR_OUT_OF_MEMORY, leaves no handle and no
device memory behind, and the next create succeeds; a refused set_preprocess upload leaves
the handle usable; a refused Normalizer scratch fails the predict with OUT_OF_MEMORY and the
next predict (limit lifted) is correct.  No kernel runs in a failing call."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import assert_scores, oracle_predict, to_dev
from synth import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def test_create_out_of_memory_leaves_nothing(monkeypatch):
    import torch
    w = make_workload("gbdt_d6", 2000)
    with B.Forest(w.forest):   # the library's code objects and first-use state are loaded
        pass
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    # the packed forest (~380 KB) is refused after the small per-class arrays were allocated
    monkeypatch.setenv("BRIDGER_TEST_ALLOC_LIMIT", "100000")
    for _ in range(50):
        with pytest.raises(B.BridgerError) as e:
            B.Forest(w.forest)
        assert e.value.status == B.BRIDGER_ERR_OUT_OF_MEMORY
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free0 - free1 <= 4 * 1024 * 1024, f"{(free0 - free1) / 1024:.0f} KiB of device memory kept"
    monkeypatch.delenv("BRIDGER_TEST_ALLOC_LIMIT")
    X = w.X()
    with B.Forest(w.forest) as f:
        got = f.predict(to_dev(X))
        torch.cuda.synchronize()
        ref, _ = oracle_predict(w.forest, X)
        assert_scores(got.cpu().numpy(), ref, "create after refused creates")


def test_preprocess_and_normalizer_out_of_memory(monkeypatch):
    import torch
    from oracle import preprocess as P
    w = make_workload("gbdt_d6", 3000)
    X = w.X()
    Xd = to_dev(X)
    F = w.n_features
    with B.Forest(w.forest) as f:
        # the scaler's parameters (F doubles each) are refused: the handle keeps predicting
        monkeypatch.setenv("BRIDGER_TEST_ALLOC_LIMIT", "64")
        with pytest.raises(B.BridgerError) as e:
            f.set_preprocess(B.BRIDGER_PRE_MINMAX, np.ones(F), np.zeros(F))
        assert e.value.status == B.BRIDGER_ERR_OUT_OF_MEMORY
        monkeypatch.delenv("BRIDGER_TEST_ALLOC_LIMIT")
        ref, _ = oracle_predict(w.forest, X)
        assert_scores(f.predict(Xd).cpu().numpy(), ref, "after a refused set_preprocess")
        a, b = np.full(F, 0.5), np.full(F, 0.25)
        f.set_preprocess(B.BRIDGER_PRE_MINMAX, a, b)
        ref_mm, _ = oracle_predict(w.forest, P.apply(P.MINMAX, a, b, X))
        assert_scores(f.predict(Xd).cpu().numpy(), ref_mm, "MinMax after a refused upload")
        # the Normalizer's row norms (8 bytes per row) are refused: predict fails, output kept
        f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)
        out = torch.full((X.shape[0], 1), -3.0, device="cuda")
        monkeypatch.setenv("BRIDGER_TEST_ALLOC_LIMIT", "1000")
        with pytest.raises(B.BridgerError) as e:
            f.predict(Xd, out)
        assert e.value.status == B.BRIDGER_ERR_OUT_OF_MEMORY
        torch.cuda.synchronize()
        assert torch.all(out == -3.0)
        # the allocation-free entry point needs no allocation: the limit does not affect it
        B.bridger_forest_predict_noalloc(f.handle, Xd.data_ptr(), X.shape[0], F, out.data_ptr(),
                                         torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ref_n, _ = oracle_predict(w.forest, P.apply(P.NORMALIZE, None, None, X))
        assert_scores(out.cpu().numpy(), ref_n, "allocation-free predict under the limit")
        monkeypatch.delenv("BRIDGER_TEST_ALLOC_LIMIT")
        assert_scores(f.predict(Xd).cpu().numpy(), ref_n, "Normalizer after a refused scratch")
