"""Build libopd.so in place: hand-written HIP for gfx950 plus the C-ABI layer."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libopd.so")
SOURCES = [os.path.join(CSRC, "opd_kernels.hip"), os.path.join(CSRC, "opd_cache_kernels.hip"),
           os.path.join(CSRC, "opd_diag_kernels.hip"), os.path.join(CSRC, "opd_noalloc.hip"),
           os.path.join(CSRC, "opd_api.cpp")]
HEADERS = [os.path.join(CSRC, "opd_internal.h"), os.path.join(CSRC, "opd_device.h"),
           os.path.join(ROOT, "include", "opd.h")]

# -packed-fp32-ops: no v_pk_* fp32 arithmetic in device code.
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++20", "-fPIC", "-shared",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-Wall", "-Wno-unused-variable", "-Wno-unused-but-set-variable"]


def build(force: bool = True, extra_flags=()) -> str:
    """Compile every source into libopd.so (always, unless force=False and it is current)."""
    if not force and os.path.exists(LIB):
        t = os.path.getmtime(LIB)
        if all(os.path.getmtime(p) <= t for p in SOURCES + HEADERS):
            return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["hipcc", *HIPCC_FLAGS, *extra_flags, "-I", os.path.join(ROOT, "include"), "-o", tmp,
           *SOURCES]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building libopd.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
