"""Build libios.so (host C++ + gfx950 HIP kernels) in-tree with hipcc.

    python paper_2011_01302_amd/build.py

Objects go to ``_build/`` at the repository root; the shared library is
written next to this file so that it travels with the source tree.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libios.so")
BUILD = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result"]
# device code: gfx950 only, packed fp32 arithmetic disabled; the stage kernel's
# first three argument words (table pointer and size) preloaded into SGPRs
DEVICE = ["-x", "hip", f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
          "-packed-fp32-ops", "-munsafe-fp-atomics", "-mllvm", "-amdgpu-kernarg-preload-count=3"]
# the stage kernel variants build as separate translation units, in parallel
SOURCES = ["stage_kernel_full.hip", "stage_kernel_full_persist.hip", "stage_kernel_sep.hip",
           "stage_kernel_sep_persist.hip", "stage_kernel_seprow.hip", "stage_kernel_seprow_persist.hip",
           "stage_kernel_pipe.hip", "stage_kernel_pipe_persist.hip", "stage_kernel_light.hip",
           "stage_kernel_light_persist.hip",
           "noalloc.hip", "graph.cpp", "sched.cpp", "exec.cpp", "api.cpp", "stage_launch.cpp"]


def _compile(src: str) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(BUILD, src + ".o")
    # host sources are plain C++ against the HIP runtime headers (no device pass)
    cmd = [HIPCC] + COMMON + (DEVICE if src.endswith(".hip") else ["-x", "c++", "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]) + \
        ["-c", path, "-o", obj]
    subprocess.check_call(cmd)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source and link libios.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp%d" % os.getpid()
    link = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    subprocess.check_call(link)
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
