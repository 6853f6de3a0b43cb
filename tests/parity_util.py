"""Shared helpers for the parity tests: run the HIP path through the C ABI and compare with
the CPU oracle on the same seeded inputs."""
from __future__ import annotations

import numpy as np

import oracle
import paper_2405_12491_amd as B

# The tolerance for float scores: |gpu - oracle| <= ATOL + RTOL * |oracle|.
RTOL = 1e-5
ATOL = 1e-6


def close_mask(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    gpu = np.asarray(gpu, np.float64)
    both_nan = np.isnan(gpu) & np.isnan(ref)
    same_inf = np.isinf(ref) & (gpu == ref)
    with np.errstate(invalid="ignore"):
        ok = np.abs(gpu - ref) <= ATOL + RTOL * np.abs(ref)
    return ok | both_nan | same_inf


def assert_scores(gpu: np.ndarray, ref: np.ndarray, what: str = ""):
    ok = close_mask(gpu, ref)
    if not ok.all():
        bad = np.argwhere(~ok)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {ok.size} scores out of tolerance; first at "
                             f"{i}: gpu {gpu[i]!r} oracle {ref[i]!r}")


def assert_leaves(gpu: np.ndarray, ref: np.ndarray, what: str = ""):
    if not np.array_equal(gpu, ref):
        bad = np.argwhere(gpu != ref)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {gpu.size} leaf ids differ; first at {i}: "
                             f"gpu {gpu[i]} oracle {ref[i]}")


def to_dev(X: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(X, np.float32)).cuda()


def gpu_predict(forest: B.Forest, Xd, leaves: bool = False):
    import torch
    out = forest.predict_leaves(Xd) if leaves else forest.predict(Xd)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def oracle_predict(model, X: np.ndarray, leaves: bool = False, threads: int = 8):
    out, lv, _ = oracle.predict(model, X, want_leaves=leaves, threads=threads)
    return out, lv


def check_parity(model, X: np.ndarray, kernel: int, what: str, exact_sum: bool = False,
                 Xd=None, forest: B.Forest | None = None):
    """Scores within tolerance and leaf ids bit-exact for every row of X."""
    own = forest is None
    if own:
        forest = B.Forest(model)
    try:
        forest.kernel = kernel
        if Xd is None:
            Xd = to_dev(X)
        ref, ref_lv = oracle_predict(model, X, leaves=True)
        got = gpu_predict(forest, Xd)
        assert_scores(got, ref, what + " scores")
        if exact_sum:
            assert np.array_equal(got, ref.astype(np.float32)), what + " not bit-identical"
        got_lv = gpu_predict(forest, Xd, leaves=True)
        assert_leaves(got_lv, ref_lv, what + " leaves")
    finally:
        if own:
            forest.close()


# Labels: where the oracle's top two values lie within TIE (relative) of each other, different
# summation orders may legitimately split them, and any class that close to the top is accepted.
TIE = 1e-12


def check_labels(got, ref, what):
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
