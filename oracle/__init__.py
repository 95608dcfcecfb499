"""CPU oracle for the dense matrix-vector family -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (``paper_2512_22147_amd``)
never imports it and shares no code with it.

Contents
--------
* ``matvec``, ``matvec_t``, ``ata_x``, ``bicg``, ``axpby_mv``: fp64 plain-loop
  definitions (``oracle.c``), inputs promoted exactly to fp64, one output
  element summed by one thread in ascending index order.  The paper names these
  kernels (ATAX, BICG, GESUMMV in Tables 1-2, Sec. 4.2) without defining them;
  the textbook definitions are used.
* ``gemver``: GEMVER (named in Tables 1-2) as the BLAS Technical Forum
  standard defines it: Ahat = A + u1 v1^T + u2 v2^T, x = beta Ahat^T y + z,
  w = alpha Ahat x.
* ``reduce_sum``, ``vector_add``: the sum of a vector and the elementwise sum
  of two vectors (the "reduction" and "vectoradd" samples of Table 3), fp64.
* ``trimmed_mean``: Eq. 3 of Sec. 3.2 -- sort the R samples ascending, drop the
  k lowest and k highest, average the remaining R - 2k; only defined for
  R > 2k.
* ``fe_error`` / ``fe_pass``: the functional-equivalence test of Eq. 4.  The
  paper only asks that outputs agree; the metric taken for that is the
  normwise relative error max_i |out_i - ref_i| / max_i |ref_i|; any
  non-finite output fails; an all-zero reference demands an all-zero output.
* ``select_next`` : Eqs. 4-5 -- among the candidates that pass FE, the one with
  the smallest trimmed-mean time becomes the next baseline.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared", "-std=c11"]


def build(source: str = SOURCE, out: str = LIB_PATH, verbose: bool = False) -> str:
    """Compile the oracle with gcc.  Building the checker is not using it."""
    cmd = ["gcc", *CFLAGS, source, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


class Oracle:
    """Binding to one build of ``oracle.c`` (tests may load altered copies)."""

    def __init__(self, lib_path: str = LIB_PATH):
        if not os.path.exists(lib_path):
            raise RuntimeError(f"{lib_path} is not built; run oracle.build()")
        lib = ctypes.CDLL(lib_path)
        i64, vp, d = ctypes.c_int64, ctypes.c_void_p, ctypes.c_double
        lib.oracle_matvec.argtypes = [i64, i64, vp, vp, vp]
        lib.oracle_matvec_t.argtypes = [i64, i64, vp, vp, vp]
        lib.oracle_ata_x.argtypes = [i64, i64, vp, vp, vp, vp]
        lib.oracle_bicg.argtypes = [i64, i64, vp, vp, vp, vp, vp]
        lib.oracle_axpby_mv.argtypes = [i64, i64, d, vp, d, vp, vp, vp]
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_reduce_sum.argtypes = [i64, vp]
        lib.oracle_reduce_sum.restype = d
        lib.oracle_vector_add.argtypes = [i64, vp, vp, vp]
        lib.oracle_gemver.argtypes = [i64, i64, d, d, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        self.lib = lib
        self.path = lib_path

    def num_threads(self) -> int:
        return int(self.lib.oracle_num_threads())

    @staticmethod
    def _shape(A):
        if A.ndim != 2:
            raise ValueError("A must be 2-D (m, n)")
        return A.shape

    def matvec(self, A, x) -> np.ndarray:
        A, x = _f64(A), _f64(x)
        m, n = self._shape(A)
        assert x.shape == (n,)
        y = np.empty(m)
        self.lib.oracle_matvec(m, n, A.ctypes.data, x.ctypes.data, y.ctypes.data)
        return y

    def matvec_t(self, A, w) -> np.ndarray:
        A, w = _f64(A), _f64(w)
        m, n = self._shape(A)
        assert w.shape == (m,)
        z = np.empty(n)
        self.lib.oracle_matvec_t(m, n, A.ctypes.data, w.ctypes.data, z.ctypes.data)
        return z

    def ata_x(self, A, x):
        """Returns (y, t) with t = A x in fp64 and y = A^T t."""
        A, x = _f64(A), _f64(x)
        m, n = self._shape(A)
        assert x.shape == (n,)
        t = np.empty(m)
        y = np.empty(n)
        self.lib.oracle_ata_x(m, n, A.ctypes.data, x.ctypes.data, t.ctypes.data, y.ctypes.data)
        return y, t

    def bicg(self, A, p, r):
        """Returns (q, s) with q = A p and s = A^T r."""
        A, p, r = _f64(A), _f64(p), _f64(r)
        m, n = self._shape(A)
        assert p.shape == (n,) and r.shape == (m,)
        q = np.empty(m)
        s = np.empty(n)
        self.lib.oracle_bicg(m, n, A.ctypes.data, p.ctypes.data, r.ctypes.data,
                             q.ctypes.data, s.ctypes.data)
        return q, s

    def axpby_mv(self, alpha, A, beta, B, x) -> np.ndarray:
        """y = alpha A x + beta B x.  alpha and beta are taken as given: pass
        the element-type values (e.g. float32(1.2)) to model an fp32 run."""
        A, B, x = _f64(A), _f64(B), _f64(x)
        m, n = self._shape(A)
        assert B.shape == (m, n) and x.shape == (n,)
        y = np.empty(m)
        self.lib.oracle_axpby_mv(m, n, float(alpha), A.ctypes.data, float(beta),
                                 B.ctypes.data, x.ctypes.data, y.ctypes.data)
        return y


    def gemver(self, alpha, beta, A, u1, v1, u2, v2, y, z):
        """Returns (Ahat, x, w).  alpha, beta are taken as given (pass the
        element-type values to model an fp32 run)."""
        A = _f64(A)
        m, n = self._shape(A)
        u1, u2, y = _f64(u1), _f64(u2), _f64(y)
        v1, v2, z = _f64(v1), _f64(v2), _f64(z)
        assert u1.shape == u2.shape == y.shape == (m,) and v1.shape == v2.shape == z.shape == (n,)
        Ahat = np.empty((m, n))
        x = np.empty(n)
        w = np.empty(m)
        self.lib.oracle_gemver(m, n, float(alpha), float(beta), A.ctypes.data, u1.ctypes.data,
                               v1.ctypes.data, u2.ctypes.data, v2.ctypes.data, y.ctypes.data,
                               z.ctypes.data, Ahat.ctypes.data, x.ctypes.data, w.ctypes.data)
        return Ahat, x, w

    def reduce_sum(self, x) -> float:
        x = _f64(x).ravel()
        return float(self.lib.oracle_reduce_sum(x.size, x.ctypes.data))

    def vector_add(self, a, b) -> np.ndarray:
        a, b = _f64(a).ravel(), _f64(b).ravel()
        assert a.shape == b.shape
        c = np.empty(a.size)
        self.lib.oracle_vector_add(a.size, a.ctypes.data, b.ctypes.data, c.ctypes.data)
        return c


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def matvec(A, x):
    return default().matvec(A, x)


def matvec_t(A, w):
    return default().matvec_t(A, w)


def ata_x(A, x):
    return default().ata_x(A, x)


def bicg(A, p, r):
    return default().bicg(A, p, r)


def axpby_mv(alpha, A, beta, B, x):
    return default().axpby_mv(alpha, A, beta, B, x)


def gemver(alpha, beta, A, u1, v1, u2, v2, y, z):
    return default().gemver(alpha, beta, A, u1, v1, u2, v2, y, z)


def reduce_sum(x):
    return default().reduce_sum(x)


def vector_add(a, b):
    return default().vector_add(a, b)


def elem_scalar(v: float, dtype) -> float:
    """A scalar as the element type holds it, promoted back to fp64."""
    return float(np.dtype(dtype).type(v))


# ---------------------------------------------------------------------------
# Harness definitions (Sec. 3.2).
# ---------------------------------------------------------------------------

def trimmed_mean(samples, k: int) -> float:
    """Eq. 3: mean of the sorted samples T_(k+1) .. T_(R-k); requires R > 2k.

    The kept samples are summed in ascending order."""
    R = len(samples)
    if k < 0 or R <= 2 * k:
        raise ValueError("Eq. 3 needs R > 2k and k >= 0")
    s = sorted(float(v) for v in samples)
    total = 0.0
    for i in range(k, R - k):
        total += s[i]
    return total / (R - 2 * k)


def fe_error(out, ref) -> float:
    """Normwise relative error max|out - ref| / max|ref| (inf if any output is
    not finite; 0 or inf for an all-zero reference)."""
    out = np.asarray(out, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    if out.shape != ref.shape:
        raise ValueError("shape mismatch")
    if out.size == 0:
        return 0.0
    worst = 0.0
    for o in out:
        if not math.isfinite(o):
            return math.inf
    scale = 0.0
    for r in ref:
        scale = max(scale, abs(r))
    for o, r in zip(out, ref):
        worst = max(worst, abs(o - r))
    if scale == 0.0:
        return 0.0 if worst == 0.0 else math.inf
    return worst / scale


def fe_pass(out, ref, tol: float) -> bool:
    """Eq. 4's FE predicate under the normwise reading."""
    return fe_error(out, ref) <= tol


def select_next(candidates):
    """Eqs. 4-5: ``candidates`` is a sequence of (name, trimmed_mean, fe_ok).

    Returns the name of the fastest FE-passing candidate (first one on ties),
    or None when the feasible set is empty."""
    best = None
    for name, t, ok in candidates:
        if not ok:
            continue
        if best is None or t < best[1]:
            best = (name, t)
    return None if best is None else best[0]
