"""Seeded synthetic inputs for the dense matrix-vector MEPs (Sec. 3.1.2, Eq. 2).

The paper's Input Data Generator produces repeatable inputs that match a
kernel's input pattern while keeping the data size S_data under a bound S_max.
This module is that generator for the matrix-vector family.  It only draws
numbers (SplitMix64 in counter form, see ``mep_datagen.c``) and describes the
workloads; it holds none of the matrix-vector arithmetic, so the GPU path and
the CPU oracle can both be fed from it without sharing any computation.

Every array is generated on the host, so both sides see identical bits.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmep_datagen.so")
SOURCE = os.path.join(_HERE, "mep_datagen.c")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the generator with gcc (no HIP involved)."""
    import subprocess

    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           SOURCE, "-o", LIB_PATH + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        lib = ctypes.CDLL(LIB_PATH)
        u64, i64, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p
        lib.mep_dg_bits.argtypes = [u64, u64, u64, i64, vp]
        for name in ("uniform", "normal", "ternary"):
            for t in ("f32", "f64"):
                getattr(lib, f"mep_dg_{name}_{t}").argtypes = [u64, u64, u64, i64, vp]
        _lib = lib
    return _lib


def bits(seed: int, array_id: int, count: int, first: int = 0) -> np.ndarray:
    """Raw SplitMix64 words bits(seed, array_id, first + k), k < count."""
    out = np.empty(int(count), dtype=np.uint64)
    _load().mep_dg_bits(seed, array_id, first, int(count), out.ctypes.data)
    return out


def _draw(kind: str, seed: int, array_id: int, shape, dtype, first: int = 0) -> np.ndarray:
    dtype = np.dtype(dtype)
    if dtype == np.float32:
        suffix = "f32"
    elif dtype == np.float64:
        suffix = "f64"
    else:
        raise ValueError(f"unsupported dtype {dtype}")
    out = np.empty(shape, dtype=dtype)
    if first < 0:
        raise ValueError("first must be >= 0")
    getattr(_load(), f"mep_dg_{kind}_{suffix}")(seed, array_id, first, out.size, out.ctypes.data)
    return out


def uniform(seed: int, array_id: int, shape, dtype=np.float32, first: int = 0) -> np.ndarray:
    """i.i.d. uniform[-1, 1) values, exact in the element type.  ``first``:
    counter of the first element, so that pieces of one large array can be
    drawn one at a time (elements first, first + 1, ... of array array_id)."""
    return _draw("uniform", seed, array_id, shape, dtype, first)


def normal(seed: int, array_id: int, shape, dtype=np.float32, first: int = 0) -> np.ndarray:
    """i.i.d. normal(0, 1) values (Box-Muller in fp64, rounded to dtype)."""
    return _draw("normal", seed, array_id, shape, dtype, first)


def ternary(seed: int, array_id: int, shape, dtype=np.float32, first: int = 0) -> np.ndarray:
    """i.i.d. values in {-1, 0, 1}; every sum of products of them is an
    integer, so results are exact in any summation order while partial sums
    stay below 2^24 (fp32) or 2^53 (fp64)."""
    return _draw("ternary", seed, array_id, shape, dtype, first)


# ---------------------------------------------------------------------------
# Workload catalogue.  Arrays are numbered in the order each workload lists
# them; that number is the SplitMix64 array id.
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    name: str
    op: str               # "ata_x" | "bicg" | "axpby_mv" | "matvec" | "matvec_t" | "gemver"
    #                       | "reduce_sum" | "vector_add"
    m: int
    n: int
    seed: int
    dist: str             # "uniform" | "normal" | "abs_uniform" (|uniform|, on [0, 1])
    arrays: tuple         # (name, length-or-shape) in generation order
    alpha: float = 0.0
    beta: float = 0.0
    note: str = ""
    dtypes: tuple = field(default=("f32",))

    def data_bytes(self, dtype) -> int:
        """S_data of Eq. 2: bytes of generated input."""
        es = np.dtype(dtype).itemsize
        tot = 0
        for _, shp in self.arrays:
            tot += int(np.prod(shp)) * es
        return tot


WORKLOADS = {
    "ata_x_1024": Workload(
        "ata_x_1024", "ata_x", 1024, 1024, 0, "uniform",
        (("A", (1024, 1024)), ("x", (1024,))),
        note="fused y = A^T (A x), fp32, small parity case"),
    "bicg_4096": Workload(
        "bicg_4096", "bicg", 4096, 4096, 1, "uniform",
        (("A", (4096, 4096)), ("p", (4096,)), ("r", (4096,))),
        note="paired q = A p and s = A^T r sharing one read of A, fp32"),
    "axpby_mv_8192": Workload(
        "axpby_mv_8192", "axpby_mv", 8192, 8192, 2, "normal",
        (("A", (8192, 8192)), ("B", (8192, 8192)), ("x", (8192,))),
        alpha=1.5, beta=1.2,
        note="scaled sum y = alpha A x + beta B x, fp32"),
    "ata_x_16384": Workload(
        "ata_x_16384", "ata_x", 16384, 16384, 3, "uniform",
        (("A", (16384, 16384)), ("x", (16384,))),
        note="fused y = A^T (A x), fp32 (1 GiB) and fp64 (2 GiB), headline",
        dtypes=("f32", "f64")),
    "reduce_sum_256m": Workload(
        "reduce_sum_256m", "reduce_sum", 1, 1 << 28, 5, "abs_uniform",
        (("x", (1 << 28,)),),
        note="s = sum of x, fp32 (1 GiB): the 'reduction' sample of Table 3; non-negative terms, "
             "so the sum does not cancel and a relative error of 1e-4 bounds it tightly"),
    "vector_add_256m": Workload(
        "vector_add_256m", "vector_add", 1, 1 << 28, 6, "uniform",
        (("a", (1 << 28,)), ("b", (1 << 28,))),
        note="c = a + b, fp32 (2 x 1 GiB in, 1 GiB out): the 'vectoradd' sample of Table 3"),
    "gemver_16384": Workload(
        "gemver_16384", "gemver", 16384, 16384, 7, "uniform",
        (("A", (16384, 16384)), ("u1", (16384,)), ("v1", (16384,)), ("u2", (16384,)),
         ("v2", (16384,)), ("y", (16384,)), ("z", (16384,))),
        alpha=1.5, beta=1.2,
        note="rank-2 update stored, then two products over it, fp32 (1 GiB read, written, read)"),
    "matvec_t_1m_x_64": Workload(
        "matvec_t_1m_x_64", "matvec_t", 1048576, 64, 4, "uniform",
        (("A", (1048576, 64)), ("w", (1048576,))),
        note="tall-skinny z = A^T w, fp32"),
}


def make_inputs(workload: Workload | str, dtype=np.float32) -> dict:
    """Generate every array of a workload, in its listed order."""
    if isinstance(workload, str):
        workload = WORKLOADS[workload]
    draw = normal if workload.dist == "normal" else uniform
    out = {}
    for aid, (name, shp) in enumerate(workload.arrays):
        out[name] = draw(workload.seed, aid, shp, dtype)
        if workload.dist == "abs_uniform":
            np.abs(out[name], out=out[name])  # exact: only the sign bit changes
    return out
