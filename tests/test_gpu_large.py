"""Matrices past the 32-bit limits: more than 2^32 bytes and, for fp32, more
than 2^31 elements, so every byte and element offset of the kernels, the
column reduce and the host planning needs 64 bits.

The matrices are drawn in row pieces by the seeded generator (each piece
from its first element's counter, bit for bit the whole draw) and uploaded
piece by piece.  Every row output (A x, BICG's q, GESUMMV, ATAX's t) is one
ascending fp64 sum per row in the oracle, so it is formed here from the same
pieces; column outputs (ATAX's y = A^T t with t kept in fp64, BICG's s =
A^T r) are checked on sampled columns, as the oracle's column sums over those
columns of A, so no fp64 copy of a whole matrix is needed.  The normwise
error of a sampled output is taken over the sampled entries.
"""
import numpy as np
import pytest

import oracle
from tests.gpu_cases import TOL, normwise

pytestmark = pytest.mark.gpu

# (dtype, m, n): 65600 x 32768 fp32 = 2,149,580,800 elements (8.6 GB per
# matrix, two for GESUMMV); 33000 x 16384 fp64 = 4.3 GB per matrix; and
# 33000 x 16383 fp64, whose rows are not 16-byte aligned (the element-wise
# path, over two column panels)
CASES = [("f32", 65600, 32768), ("f64", 33000, 16384), ("f64", 33000, 16383)]


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dts,m,n", CASES, ids=[f"{d}-{m}x{n}" for d, m, n in CASES])
def test_every_matrix_op_beyond_32_bit_offsets(dts, m, n):
    """ATAX (y sampled, t every row), y = A x, BICG (q every row, s sampled)
    and GESUMMV (every row) on one matrix past the 32-bit limits."""
    import torch

    from paper_2512_22147_amd import datagen, mep

    dt = np.float32 if dts == "f32" else np.float64
    tdt = torch.float32 if dts == "f32" else torch.float64
    es = np.dtype(dt).itemsize
    assert m * n * es > 2 ** 32
    if dts == "f32":
        assert m * n > 2 ** 31
    dev = torch.device("cuda:0")
    seed = 21
    alpha, beta = oracle.elem_scalar(1.5, dt), oracle.elem_scalar(1.2, dt)
    # array numbers as in the parity tests: A 0, x 1, w 2, B 3
    x = datagen.uniform(seed, 1, (n,), dt)
    w = datagen.uniform(seed, 2, (m,), dt)
    rng = np.random.default_rng(seed)
    cols = np.unique(np.concatenate([[0, 1, n - 2, n - 1], rng.choice(n, 252, replace=False)]))

    A = torch.empty((m, n), dtype=tdt, device=dev)
    B = torch.empty((m, n), dtype=tdt, device=dev)
    t_ref = np.empty(m, dtype=np.float64)
    g_ref = np.empty(m, dtype=np.float64)
    a_cols = np.empty((m, cols.size), dtype=dt)
    rows = max(1, (1 << 28) // (n * es))  # 256 MiB pieces
    for r0 in range(0, m, rows):
        r1 = min(m, r0 + rows)
        pa = datagen.uniform(seed, 0, (r1 - r0, n), dt, first=r0 * n)
        pb = datagen.uniform(seed, 3, (r1 - r0, n), dt, first=r0 * n)
        A[r0:r1].copy_(torch.from_numpy(pa))
        B[r0:r1].copy_(torch.from_numpy(pb))
        t_ref[r0:r1] = oracle.matvec(pa, x)
        g_ref[r0:r1] = oracle.axpby_mv(alpha, pa, beta, pb, x)
        a_cols[r0:r1] = pa[:, cols]
        del pa, pb
    y_ref = oracle.matvec_t(a_cols, t_ref)  # ATAX: t kept in fp64
    s_ref = oracle.matvec_t(a_cols, w)

    xg = torch.from_numpy(x).to(dev)
    wg = torch.from_numpy(w).to(dev)
    t = torch.empty(m, dtype=tdt, device=dev)
    y = mep.mep_ata_x(A, xg, t=t)
    yv = mep.mep_matvec(A, xg)
    s, q = mep.mep_matvec_t(A, wg, p=xg)
    g = mep.mep_axpby_mv(1.5, A, 1.2, B, xg)
    torch.cuda.synchronize()
    tol = TOL[dt]
    for name, got, ref in (("ATAX t", t.cpu().numpy(), t_ref),
                           ("ATAX y (sampled columns)", y.cpu().numpy()[cols], y_ref),
                           ("A x", yv.cpu().numpy(), t_ref),
                           ("BICG q", q.cpu().numpy(), t_ref),
                           ("BICG s (sampled columns)", s.cpu().numpy()[cols], s_ref),
                           ("GESUMMV", g.cpu().numpy(), g_ref)):
        err = normwise(got, ref)
        assert err <= tol, f"{name}: normwise error {err:.3e} > {tol:.0e}"
    del A, B, t, y, yv, s, q, g
