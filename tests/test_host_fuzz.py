"""The host side of the library (validation, packing, planning, queries) under AddressSanitizer
and UndefinedBehaviorSanitizer: bridger_host.cpp is rebuilt with the sanitizers on its host code
and driven by tests/host_fuzz.cpp over random and corrupted forests on host-only handles."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer"]


def test_host_code_under_sanitizers(tmp_path):
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    kernel_objs = [o for o in glob.glob(os.path.join(ROOT, "paper_2405_12491_amd", "_build", "*.o"))
                   if not os.path.basename(o).startswith("bridger_host")]
    if not kernel_objs:
        pytest.skip("kernel objects not built (run __graft_entry__.build())")
    common = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
              "-I", os.path.join(ROOT, "include"),
              "-I", os.path.join(ROOT, "paper_2405_12491_amd", "csrc"),
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    host_o, fuzz_o, exe = (str(tmp_path / n) for n in ("host.o", "fuzz.o", "fuzz"))
    subprocess.run([HIPCC, *common, *SAN, "-c", "-x", "hip",
                    os.path.join(ROOT, "paper_2405_12491_amd", "csrc", "bridger_host.cpp"),
                    "-o", host_o], check=True, capture_output=True)
    subprocess.run([HIPCC, *common, *SAN, "-c", "-x", "hip",
                    os.path.join(ROOT, "tests", "host_fuzz.cpp"), "-o", fuzz_o],
                   check=True, capture_output=True)
    # link with the host compiler (the sanitizer runtimes are host libraries)
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(HIPCC)))
    clangxx = os.path.join(rocm, "llvm", "bin", "clang++")
    subprocess.run([clangxx, "-fsanitize=address,undefined", "-o", exe, fuzz_o, host_o,
                    *kernel_objs, "-L" + os.path.join(rocm, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + os.path.join(rocm, "lib")], check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, "2000"], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert out.strip().startswith("ok "), out[-2000:]
