"""Build step for the HIP library ``libedkm.so`` (gfx950), in-tree."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("edkm_kernels.hip", "edkm_api.hip")]
OUT = os.path.join(HERE, "libedkm.so")
# Diagnostics build: the same library with per-block timeline stamps
# (-DEDKM_BLOCK_STAMPS, include/edkm_stamps.h); load it with EDKM_LIBRARY.
OUT_STAMPS = os.path.join(HERE, "libedkm_stamps.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Werror=uninitialized",
    # no packed-fp32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]


def build_library(out: str = OUT, extra=()) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc, *HIPCC_FLAGS, *extra, "-o", tmp, *SOURCES]
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


def build_stamps(out: str = OUT_STAMPS) -> str:
    return build_library(out, extra=("-DEDKM_BLOCK_STAMPS",))


if __name__ == "__main__":
    print(build_library())
    print(build_stamps())
