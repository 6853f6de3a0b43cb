"""Compile the HIP library (gfx950) in-tree: paper_2405_12491_amd/libbridger.so.

Each source is compiled to an object in parallel under paper_2405_12491_amd/_build, then the
objects are linked into the shared library (written to a temporary name, then renamed).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libbridger.so")
CALIB_LIB = os.path.join(PKG, "libbridger_calib.so")
CALIB_SOURCES = [os.path.join(CSRC, "calib.hip")]
SOURCES = [os.path.join(CSRC, n) for n in
           ("bridger_host.cpp", "perfect.hip", "perfect_binned.hip", "perfect_fixed.hip",
            "perfect_global.hip", "ragged.hip", "direct.hip", "gemm.hip", "bin.hip",
            "normalize.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

ARCH = ["--offload-arch=gfx950"]
FLAGS = ARCH + [
    "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-gpu-rdc", "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, "-c", "-o", obj]
    cmd += ["-x", "hip", src] if src.endswith(".cpp") else [src]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed compiling {os.path.basename(src)}")
    return obj


def _link(objs, lib: str, verbose: bool):
    tmp = lib + ".tmp"
    cmd = [HIPCC, *ARCH, "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"linking {os.path.basename(lib)} failed")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Build libbridger.so (the prediction library) and libbridger_calib.so (the calibration
    microbenchmarks used by the benchmark); returns the prediction library's path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = SOURCES + CALIB_SOURCES
    jobs = max(1, min(len(srcs), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    _link(objs[:len(SOURCES)], LIB, verbose)
    _link(objs[len(SOURCES):], CALIB_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
