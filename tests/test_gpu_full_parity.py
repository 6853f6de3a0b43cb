"""Exhaustive full-size parity on the five benchmark workloads.

Each workload runs at its full size in the benchmark's launch configuration: one predict and
one predict_leaves call over the whole batch (the plan the benchmark times), with the rows
resident on the device.  Every row's scores and every (row, tree) leaf id are then compared
with the multi-threaded oracle, in row chunks so that host memory stays near a few GB (the
ragged workload alone has 16 GB of leaf ids).  The operators whose results must agree are the
comparison, conditional and aggregation categories of the classical operator representation
(Sec. 4.2; Table 4: less_equal, where, sum/mean) and the link functions (exp, divide, max).

Scores: |gpu - oracle| <= 1e-6 + 1e-5 |oracle|; leaf ids bit-exact.
"""
import os
import time

import numpy as np
import pytest

import paper_2405_12491_amd as B
from parity_util import assert_leaves, assert_scores, oracle_predict
from synth import CONFIGS, make_workload, x_rows_threaded

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CHUNK_ROWS = 1 << 18


def _threads():
    # the machine's CPU share for one GPU is 16 threads, whatever the affinity mask shows
    return max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()
    yield


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", list(CONFIGS))
def test_full_size_exhaustive(name):
    import torch
    w = make_workload(name)
    f_ = w.forest
    n, F, T, K = w.n_rows, w.n_features, f_.n_trees, f_.n_classes
    th = _threads()
    t0 = time.perf_counter()
    print(f"[exhaustive] {name}: {n} rows x {F} features, {T} trees, {K} outputs; "
          f"oracle on {th} threads, chunks of {CHUNK_ROWS} rows", flush=True)
    Xd = torch.empty((n, F), dtype=torch.float32, device="cuda")
    host = []
    for a in range(0, n, CHUNK_ROWS):
        b = min(n, a + CHUNK_ROWS)
        Xc = x_rows_threaded(w.seed, w.x_kind, F, a, b, th, **w.x_params)
        Xd[a:b].copy_(torch.from_numpy(Xc))
        host.append((a, b, Xc))
    print(f"[exhaustive] {name}: X built ({time.perf_counter() - t0:.1f} s)", flush=True)
    n_scores = n_leaves = 0
    with B.Forest(f_) as f:
        plan = f.plan(n)
        print(f"[exhaustive] {name}: kernel={B.KERNEL_NAMES[f.kernel]} plan={plan}", flush=True)
        out = f.predict(Xd)                  # the benchmark's call: the whole batch at once
        lv = f.predict_leaves(Xd)
        torch.cuda.synchronize()
        print(f"[exhaustive] {name}: GPU done ({time.perf_counter() - t0:.1f} s)", flush=True)
        for i, (a, b, Xc) in enumerate(host):
            ref, ref_lv = oracle_predict(f_, Xc, leaves=True, threads=th)
            got = out[a:b].cpu().numpy()
            assert_scores(got, ref, f"{name} rows [{a}, {b}) scores")
            assert np.all(np.isfinite(got))
            got_lv = lv[a:b].cpu().numpy()
            assert_leaves(got_lv, ref_lv, f"{name} rows [{a}, {b}) leaf ids")
            n_scores += got.size
            n_leaves += got_lv.size
            host[i] = None
            del ref, ref_lv, got_lv
            print(f"[exhaustive] {name}: rows [{a}, {b}) agree "
                  f"({time.perf_counter() - t0:.1f} s)", flush=True)
    del Xd, out, lv
    torch.cuda.empty_cache()
    assert n_scores == n * K and n_leaves == n * T
    print(f"[exhaustive] {name}: compared {n_scores} scores and {n_leaves} leaf ids "
          f"({n} rows), all equal within tolerance / bit-exact; "
          f"{time.perf_counter() - t0:.1f} s", flush=True)
