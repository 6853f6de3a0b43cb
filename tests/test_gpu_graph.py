"""Predictions captured in a HIP graph (torch.cuda.CUDAGraph on the launch stream): the graph is
replayed several times, with the program's own eager work (new rows written into the captured
input buffer) and synchronizations between replays, and every replay is checked against the
eager prediction on the same rows."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import assert_leaves, assert_scores, oracle_predict
from synth import make_workload, random_tiny_forest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


def _cases():
    rng = np.random.default_rng(8)
    out = []
    for name, n in (("gbdt_d6", 3000), ("dt_d3", 10_000), ("mc_gbdt_d8", 200), ("rf_d8", 1500)):
        w = make_workload(name, n)
        out.append((name, w.forest, [w.X(n)] + [x.astype(np.float32) for x in
                                                 (rng.standard_normal((n, w.n_features)),) * 1]))
    m = random_tiny_forest(rng, 30, 7, max_depth=9)
    out.append(("tiny_ragged", m, [rng.standard_normal((2000, 7)).astype(np.float32) for _ in range(2)]))
    return out


@pytest.mark.parametrize("case", range(5))
def test_predict_in_graph(case):
    import torch
    name, model, Xs = _cases()[case]
    n, F = Xs[0].shape
    Xd = torch.from_numpy(Xs[0]).cuda()
    out = torch.empty((n, model.n_classes), dtype=torch.float32, device="cuda")
    leaves = torch.empty((n, model.n_trees), dtype=torch.int32, device="cuda")
    with B.Forest(model) as f:
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            f.predict(Xd, out)           # eager first call: the kernels' one-time set-up
            f.predict_leaves(Xd, leaves)
        s.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            f.predict(Xd, out)
            f.predict_leaves(Xd, leaves)
        for rep in range(4):
            X = Xs[rep % len(Xs)] if rep < 2 else (Xs[0] * np.float32(0.5 + rep)).astype(np.float32)
            Xd.copy_(torch.from_numpy(X))        # eager work between replays
            torch.cuda.synchronize()
            out.zero_()
            leaves.zero_()
            g.replay()
            torch.cuda.synchronize()
            ref, ref_lv = oracle_predict(model, X, leaves=True)
            assert_scores(out.cpu().numpy(), ref, f"{name} replay {rep}")
            assert_leaves(leaves.cpu().numpy(), ref_lv, f"{name} replay {rep} leaves")
            eager = f.predict(Xd)
            torch.cuda.synchronize()
            assert np.array_equal(eager.cpu().numpy().view(np.uint32), out.cpu().numpy().view(np.uint32))


def test_normalizer_in_graph():
    """The Normalizer's row-norm scratch is stream-ordered (hipMallocAsync / hipFreeAsync on the
    launch stream), which a graph records as allocation nodes: replays must still match."""
    import torch
    from oracle import preprocess as P
    rng = np.random.default_rng(12)
    w = make_workload("gbdt_d6", 3000)
    X0 = w.X(3000)
    Xd = torch.from_numpy(X0).cuda()
    out = torch.empty((3000, 1), dtype=torch.float32, device="cuda")
    with B.Forest(w.forest) as f:
        f.set_preprocess(B.BRIDGER_PRE_NORMALIZE)
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            f.predict(Xd, out)
        s.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            f.predict(Xd, out)
        for rep in range(4):
            X = (rng.standard_normal(X0.shape) * (rep + 1)).astype(np.float32)
            Xd.copy_(torch.from_numpy(X))
            torch.cuda.synchronize()
            out.zero_()
            g.replay()
            torch.cuda.synchronize()
            ref, _ = oracle_predict(w.forest, P.apply(P.NORMALIZE, None, None, X))
            assert_scores(out.cpu().numpy(), ref, f"normalized replay {rep}")


@pytest.mark.parametrize("name,n", [("gbdt_d6", 3000), ("mc_gbdt_d8", 200)])
def test_binning_and_binned_predict_in_graph(name, n):
    """A serving pipeline in one graph: the binning pass writes the bins of the captured input,
    then the binned prediction reads them (two kernels, no allocation); replays with new rows
    match the oracle and an eager run bit for bit."""
    import torch
    rng = np.random.default_rng(21)
    w = make_workload(name, n)
    X0 = w.X(n)
    Xd = torch.from_numpy(X0).cuda()
    out = torch.empty((n, w.forest.n_classes), dtype=torch.float32, device="cuda")
    with B.Forest(w.forest) as f:
        q = f.bin(Xd)
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            f.bin(Xd, q)
            f.predict_binned(q, out)
        s.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            f.bin(Xd, q)
            f.predict_binned(q, out)
        for rep in range(4):
            X = (rng.standard_normal(X0.shape) * (rep + 1)).astype(np.float32) if rep else X0
            Xd.copy_(torch.from_numpy(X))
            torch.cuda.synchronize()
            out.zero_()
            g.replay()
            torch.cuda.synchronize()
            ref, _ = oracle_predict(w.forest, X)
            assert_scores(out.cpu().numpy(), ref, f"{name} binned replay {rep}")
            eager = f.predict_binned(f.bin(Xd))
            torch.cuda.synchronize()
            assert np.array_equal(eager.cpu().numpy().view(np.uint32), out.cpu().numpy().view(np.uint32))
