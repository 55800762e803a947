"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU).

libopd.so is built with both sanitizers on its host code only (every
-fsanitize flag follows -Xarch_host, so the gfx950 code is built as usual),
and the C-ABI tests (tests/test_abi.py: every argument check and error code
of every entry point, the workspace and scratch sizing, the status strings)
run against it in a child process with the sanitizer runtime preloaded.
None of those calls reaches the GPU.  Leak detection is off: the Python
interpreter and the HIP runtime hold memory until exit by design."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2606_24143_amd", "csrc")
SOURCES = ["opd_kernels.hip", "opd_cache_kernels.hip", "opd_diag_kernels.hip", "opd_noalloc.hip",
           "opd_api.cpp"]

CHILD = r"""
import sys
sys.path.insert(0, %(root)r)
sys.path.insert(0, %(tests)r)
import paper_2606_24143_amd._binding as b
b.LIB_PATH = %(lib)r
import pytest
sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", %(abi)r, "-m", "not gpu"]))
"""


def test_abi_error_paths_run_clean_under_host_sanitizers(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    runtimes = glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not os.path.exists(hipcc) or not runtimes:
        pytest.skip("hipcc or the clang sanitizer runtime not available")
    lib = str(tmp_path / "libopd.so")
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-std=c++20", "-fPIC", "-shared",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-g",
           "-Xarch_host", "-fsanitize=address",
           "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all",
           "-shared-libsan", "-o", lib] + [os.path.join(CSRC, f) for f in SOURCES]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=1800)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ, LD_PRELOAD=runtimes[0], ASAN_OPTIONS="detect_leaks=0")
    child = CHILD % {"root": ROOT, "tests": HERE, "lib": lib,
                     "abi": os.path.join(HERE, "test_abi.py")}
    run = subprocess.run([sys.executable, "-c", child], capture_output=True, text=True, env=env,
                         timeout=900)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-4000:]
    assert "passed" in run.stdout and "failed" not in run.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out
