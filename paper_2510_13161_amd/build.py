"""Build the native parts in-tree for gfx950.

* ``libmsd.so``                 the product: HIP kernels + the C ABI (include/msd.h)
* ``synth/libmsd_synth_dev.so`` device side of the synthetic-input generator
* ``synth/libmsd_synth_host.so`` host side of the synthetic-input generator

Every call recompiles. HIP code is built with packed-FP32 instructions
disabled (``-packed-fp32-ops``).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmsd.so")
INCLUDE = os.path.join(ROOT, "include")

ARCH = "gfx950"
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-function", "-I" + INCLUDE, "-I" + CSRC]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


def build_synth_host(verbose: bool = False) -> str:
    src = os.path.join(PKG, "synth", "synth_host.c")
    out = os.path.join(PKG, "synth", "libmsd_synth_host.so")
    _run(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", "-Wall", "-o", out, src],
         verbose)
    return out


def build_synth_dev(verbose: bool = False) -> str:
    src = os.path.join(PKG, "synth", "synth_dev.hip")
    out = os.path.join(PKG, "synth", "libmsd_synth_dev.so")
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", out, src], verbose)
    return out


# Per-source compiler options. gemm.hip: MFMA accumulators in architectural
# VGPRs. In the accumulator-register form the allocator let the multi-row-tile
# k-loops write each product to a different register than it read and undo
# the rotation with ~1.6 register moves per MFMA on every iteration (each
# waiting for the MFMA before it); in this form those loops have none, and
# the 3- and 5-row-tile variants fit two waves per SIMD.
SRC_FLAGS = {"gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def build_lib(verbose: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    objs = [os.path.join(BUILD_DIR, os.path.basename(s) + ".o") for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(_run, [HIPCC, *HIP_FLAGS, *SRC_FLAGS.get(os.path.basename(s), []), "-c", s,
                                 "-o", o], verbose)
                for s, o in zip(srcs, objs)]
        for f in futs:
            f.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


def build_all(verbose: bool = False) -> None:
    with cf.ThreadPoolExecutor(max_workers=3) as ex:
        futs = [ex.submit(build_synth_host, verbose), ex.submit(build_synth_dev, verbose),
                ex.submit(build_lib, verbose)]
        for f in futs:
            f.result()


if __name__ == "__main__":
    build_all(verbose="-v" in sys.argv)
