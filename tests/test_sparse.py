"""CSR rows: the densifying oracle against scipy (CPU), and GPU prediction from CSR rows
against the oracle on the densified rows."""
import numpy as np
import pytest

import paper_2405_12491_amd as B
from oracle import preprocess as P
from oracle import sparse as S
from parity_util import assert_leaves, assert_scores, oracle_predict
from synth import make_workload, random_tiny_forest


def _random_csr(rng, n, F, density, sort=True, bad_index=False):
    indptr = [0]
    indices, values = [], []
    for i in range(n):
        k = rng.binomial(F, density)
        idx = rng.choice(F, k, replace=False)
        if sort:
            idx = np.sort(idx)
        v = rng.standard_normal(k).astype(np.float32)
        if k and rng.random() < 0.05:
            v[0] = np.nan
        if bad_index and k and rng.random() < 0.1:
            idx = idx.copy()
            idx[-1] = F + 3 if rng.random() < 0.5 else -1
        indices += idx.tolist()
        values += v.tolist()
        indptr.append(len(indices))
    return (np.array(indptr, np.int64), np.array(indices, np.int32), np.array(values, np.float32))


def _sorted_csr(ip, ix, v):
    """The same rows with each row's entries in ascending index order."""
    ix2, v2 = ix.copy(), v.copy()
    for i in range(len(ip) - 1):
        o = np.argsort(ix[ip[i]:ip[i + 1]], kind="stable")
        ix2[ip[i]:ip[i + 1]] = ix[ip[i]:ip[i + 1]][o]
        v2[ip[i]:ip[i + 1]] = v[ip[i]:ip[i + 1]][o]
    return ip, ix2, v2


def test_densify_matches_scipy():
    import scipy.sparse as sp
    rng = np.random.default_rng(1)
    ip, ix, v = _random_csr(rng, 300, 40, 0.2)
    ref = sp.csr_matrix((v, ix, ip), shape=(300, 40)).toarray()
    got = S.densify(ip, ix, v, 300, 40)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(np.nan_to_num(got), np.nan_to_num(ref))
    # out-of-range indices are dropped, nothing else changes
    ip2, ix2, v2 = ip.copy(), ix.copy(), v.copy()
    ix2[0] = 99
    got2 = S.densify(ip2, ix2, v2, 300, 40)
    got[0, ix[0]] = 0.0
    assert np.array_equal(np.nan_to_num(got2), np.nan_to_num(got))


@pytest.mark.gpu
@pytest.mark.parametrize("case", ["mc_gbdt_d8", "gbdt_d6", "ragged_d12", "tiny_ragged",
                                  "tiny_ragged_chunked"])
def test_csr_prediction(case, monkeypatch):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if case.endswith("_chunked"):   # ragged trees through LDS chunks instead of global records
        monkeypatch.setenv("BRIDGER_GLOBAL", "0")
        case = case[:-len("_chunked")]
    rng = np.random.default_rng({"mc_gbdt_d8": 1, "gbdt_d6": 2, "ragged_d12": 3, "tiny_ragged": 4}[case])
    if case == "tiny_ragged":
        model = random_tiny_forest(rng, 25, 9, max_depth=8)
        n, F = 800, 9
    else:
        w = make_workload(case, {"mc_gbdt_d8": 300, "gbdt_d6": 1500, "ragged_d12": 200}[case])
        model, n, F = w.forest, w.n_rows, w.n_features
    ip, ix, v = _random_csr(rng, n, F, 0.2 if F > 100 else 0.5, sort=case != "gbdt_d6",
                            bad_index=case == "tiny_ragged")
    X = S.densify(ip, ix, v, n, F)
    d = lambda a: torch.from_numpy(a).cuda()
    with B.Forest(model) as f:
        for k in (B.BRIDGER_KERNEL_PERFECT, B.BRIDGER_KERNEL_RAGGED):
            try:
                f.kernel = k
            except B.BridgerError:
                continue
            for pre in (P.NONE, P.MINMAX, P.NORMALIZE):
                a = rng.uniform(0.5, 2.0, F) if pre == P.MINMAX else None
                b = rng.uniform(-1, 1, F) if pre == P.MINMAX else None
                f.set_preprocess(pre, a, b)
                ref, ref_lv = oracle_predict(model, P.apply(pre, a, b, X), leaves=True)
                # the row norm sums in stored order: ascending indices give the oracle's order
                cip, cix, cv = _sorted_csr(ip, ix, v) if pre == P.NORMALIZE else (ip, ix, v)
                out = f.predict_csr(d(cip), d(cix), d(cv), n)
                lv = f.predict_csr(d(cip), d(cix), d(cv), n, leaves=True)
                torch.cuda.synchronize()
                what = f"{case} csr {B.KERNEL_NAMES[k]} pre={pre}"
                assert_scores(out.cpu().numpy().astype(np.float64), ref, what)
                assert_leaves(lv.cpu().numpy(), ref_lv, what)
        f.set_preprocess(P.NONE)
        f.kernel = B.BRIDGER_KERNEL_DIRECT
        out = torch.empty((n, model.n_classes), device="cuda")
        with pytest.raises(B.BridgerError) as e:
            f.predict_csr(d(ip), d(ix), d(v), n, out=out)
        assert e.value.status == B.BRIDGER_ERR_UNSUPPORTED


@pytest.mark.gpu
def test_csr_rows_without_entries():
    """Rows that store no entry (every feature reads 0.0): the index and value arrays are empty
    and may be null; the result is the prediction of all-zero rows."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(115)
    model = random_tiny_forest(rng, 12, 3, max_depth=6)
    n = 70
    X = np.zeros((n, 3), np.float32)
    ref, ref_lv = oracle_predict(model, X, leaves=True)
    ip = torch.zeros(n + 1, dtype=torch.int64, device="cuda")
    ix = torch.empty(0, dtype=torch.int32, device="cuda")
    v = torch.empty(0, dtype=torch.float32, device="cuda")
    with B.Forest(model) as f:
        out = f.predict_csr(ip, ix, v, n)
        lv = f.predict_csr(ip, ix, v, n, leaves=True)
        torch.cuda.synchronize()
        assert_scores(out.cpu().numpy().astype(np.float64), ref, "empty csr")
        assert_leaves(lv.cpu().numpy(), ref_lv, "empty csr")
        with pytest.raises(B.BridgerError) as e:  # indptr is always needed
            B.bridger_forest_predict_csr(f._h, 0, 0, 0, n, 3, out.data_ptr(),
                                         torch.cuda.current_stream().cuda_stream)
        assert e.value.status == B.BRIDGER_ERR_INVALID_ARGUMENT
