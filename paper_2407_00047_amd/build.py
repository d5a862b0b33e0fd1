"""Build the native libraries of the package in-tree.

libqlm.so      HIP kernels + C interface (hipcc, gfx950)
libqlm_gen.so  synthetic plan generator (gcc, host C)
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LIB = os.path.join(HERE, "libqlm.so")
ARCH = "gfx950"
SOURCES = ["qlm.hip", "search.hip", "fcfs.hip", "profile.hip"]

HIP_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=" + ARCH, "-fPIC", "-shared",
    # packed fp32 instructions stay off (see the design notes)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-Wall", "-Wno-unused-function",
]


def build_hip(verbose: bool = False, extra=()) -> str:
    srcs = [os.path.join(HERE, "csrc", f) for f in SOURCES]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *HIP_FLAGS, *extra, "-o", tmp, *srcs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_all(verbose: bool = False) -> None:
    from . import workload
    workload.build_generator(force=True)
    build_hip(verbose=verbose)


if __name__ == "__main__":
    sys.path.insert(0, ROOT)
    from paper_2407_00047_amd import build as b  # noqa: E402
    b.build_all(verbose=True)
