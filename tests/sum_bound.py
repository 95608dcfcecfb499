"""Worst-case error bound of the library's sum (mep_reduce_sum), derived from
its summation depth.

Any floating-point summation whose longest chain of additions is d satisfies
|s_computed - s| <= gamma_d * sum_i |x_i|, gamma_d = d u / (1 - d u), with u
the unit roundoff (Higham, Accuracy and Stability of Numerical Algorithms,
2nd ed., Sec. 4.2: every term passes through at most d roundings).  The
oracle's reference is itself such a sum (ascending order, d = n - 1, in fp64),
so the two differ by at most the sum of their bounds.

The sum's order (include/mep.h, mep_reduce_sum): nb workgroups, nb = min(
ceil(n_v / 8192), 512) with n_v the 16-byte vectors of x (n * esize / 16), each
take one contiguous chunk of ceil(n_l / nb) loads, where n_l is n_v on the
16-byte path and n on the element-wise path (x not 16-byte aligned); the
256 lanes of a workgroup stride through the chunk, so each lane's running sum
is a chain of at most ceil(chunk / 256) additions.  What follows (the
elements of a vector, the trailing n mod VW elements, the 64-lane butterfly,
the four waves, then up to 512 partials added by slices and a pairwise tree)
adds fewer than 64 further levels; the bound takes d = ceil(chunk / 256) + 64.
"""
import math

import numpy as np

UNIT_ROUNDOFF = {np.dtype(np.float32): 2.0**-24, np.dtype(np.float64): 2.0**-53}


def sum_chunks(n: int, dt, offset: int = 0):
    """(number of workgroups, loads per workgroup chunk, elements per load)."""
    es = np.dtype(dt).itemsize
    nv = n * es // 16
    nb = max(1, min((nv + 8191) // 8192, 512))
    vw = 16 // es if (offset * es) % 16 == 0 else 1
    loads = n // vw
    return nb, -(-loads // nb), vw


def sum_depth(n: int, dt, offset: int = 0) -> int:
    _, chunk, _ = sum_chunks(n, dt, offset)
    return -(-chunk // 256) + 64


def gamma(d: int, u: float) -> float:
    return d * u / (1.0 - d * u) if d * u < 1 else math.inf


def sum_error_bound(n: int, dt, offset: int = 0) -> float:
    """Bound on |s_gpu - s_oracle| / sum |x_i| for the sum of n elements of
    dtype dt: gamma_d of the GPU's order plus gamma_(n-1) in fp64 of the
    oracle's own ascending-order sum (which dominates for fp64 inputs: the
    oracle is not exact either)."""
    d = sum_depth(n, dt, offset)
    return gamma(d, UNIT_ROUNDOFF[np.dtype(dt)]) + gamma(max(n - 1, 0), UNIT_ROUNDOFF[np.dtype(np.float64)])
