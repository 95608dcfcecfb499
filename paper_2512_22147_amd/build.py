"""Builds libmep.so (HIP, gfx950) and the input generator in-tree.

    python -m paper_2512_22147_amd.build

The HIP sources are compiled in parallel with hipcc for gfx950 only, with
packed-fp32 instructions disabled, and linked into ``libmep.so`` next to
this file.  Object files go to ``_build/`` (not tracked).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB_PATH = os.path.join(PKG, "libmep.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions in any kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]
SOURCES = ["mep_api.hip", "mep_launch_f32.hip", "mep_launch_f64.hip", "mep_launch_f32_wide.hip",
           "mep_launch_f64_wide.hip"]
HEADERS = ["mep_kernels.hpp", "mep_vector_kernels.hpp", "mep_internal.hpp", "mep_launch.inc"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature; that warning is noise
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build_mep(verbose: bool = False, jobs: int = 5) -> str:
    """Compile every HIP source for gfx950 and link libmep.so."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB_PATH + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def build(verbose: bool = False) -> None:
    from . import datagen

    datagen.build(verbose=verbose)
    build_mep(verbose=verbose)


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB_PATH)
