"""Build the native parts in-tree: libspardl.so (HIP, gfx950) and libgradgen.so
(host C, the synthetic-input generator).  Always recompiles."""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
SPARDL_SO = os.path.join(PKG, "libspardl.so")
GRADGEN_SO = os.path.join(PKG, "workloads", "libgradgen.so")
GRADGEN_DEV_SO = os.path.join(PKG, "workloads", "libgradgen_dev.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# sources of libspardl.so (csrc/): the entry points, then the kernels by stage
KERNEL_SOURCES = ("api.hip", "kernels_add.hip", "kernels_select.hip", "kernels_merge.hip", "kernels_decode.hip", "kernels_variants.hip")

HIP_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-ffp-contract=off",            # no fused multiply-add anywhere: every add is one IEEE add
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fPIC",
    "-shared",
    "-Wall",
]


def _run(cmd, verbose):
    if verbose:
        print("+", " ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build_gradgen(verbose: bool = True) -> str:
    src = os.path.join(PKG, "workloads", "gradgen.c")
    tmp = GRADGEN_SO + ".tmp"
    _run(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
          "-shared", "-Wall", src, "-o", tmp], verbose)
    os.replace(tmp, GRADGEN_SO)
    return GRADGEN_SO


def build_gradgen_dev(verbose: bool = True) -> str:
    src = os.path.join(PKG, "workloads", "gradgen_dev.hip")
    tmp = GRADGEN_DEV_SO + ".tmp"
    _run([HIPCC, *HIP_FLAGS, src, "-o", tmp], verbose)
    os.replace(tmp, GRADGEN_DEV_SO)
    return GRADGEN_DEV_SO


def build_spardl(verbose: bool = True) -> str:
    srcs = [os.path.join(CSRC, f) for f in KERNEL_SOURCES]
    tmp = SPARDL_SO + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-I", os.path.join(ROOT, "include"), *srcs, "-o", tmp], verbose)
    os.replace(tmp, SPARDL_SO)
    return SPARDL_SO


def build_all(verbose: bool = True) -> None:
    if shutil.which("gcc") is None:
        raise RuntimeError("gcc not found")
    build_gradgen(verbose)
    build_gradgen_dev(verbose)
    build_spardl(verbose)


if __name__ == "__main__":
    build_all(verbose="-q" not in sys.argv)
