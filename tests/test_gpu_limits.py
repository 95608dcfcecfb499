"""The largest sizes the library accepts, on the GPU against the oracle.

- Rows of 65535 * 8192 elements, the longest accepted, as one-row matrices
  (2 GiB fp32, 4 GiB fp64).  The plans cut them into up to 65535 column
  panels, as many as one launch holds (the element-wise path, taken by the
  fp32 row of 65535 * 8192 - 1 elements, and fp64 GESUMMV), and the column
  outputs (A^T w, BICG's s, ATAX's y, GEMVER's x) are wider than one launch
  of the column reduce covers.
- 2^30 rows of one element, the most rows accepted (4 GiB fp32).

Every op runs on each; inputs come from the seeded generator, and every
output is compared in full with the oracle's by the normwise metric, in
slices so that no fp64 temporary of a whole output is formed.
"""
import numpy as np
import pytest

from tests.gpu_cases import OPS, TOL, gpu_outputs, make_inputs, oracle_outputs

pytestmark = pytest.mark.gpu

MAX_M = 1 << 30
MAX_N = 65535 * 8192
CASES = [("f32", 1, MAX_N - 1), ("f64", 1, MAX_N), ("f32", MAX_M, 1)]


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.empty_cache()


def normwise_sliced(out, ref, piece=1 << 25):
    """max_i |out_i - ref_i| / max_i |ref_i| (inf if any out_i is not finite)."""
    out = np.ravel(out)
    ref = np.ravel(ref)
    assert out.shape == ref.shape
    worst = scale = 0.0
    for i in range(0, out.size, piece):
        o = out[i:i + piece].astype(np.float64)
        r = ref[i:i + piece].astype(np.float64)
        if not np.isfinite(o).all():
            return float("inf")
        worst = max(worst, float(np.max(np.abs(o - r))))
        scale = max(scale, float(np.max(np.abs(r))))
    if scale == 0.0:
        return 0.0 if worst == 0.0 else float("inf")
    return worst / scale


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("dts,m,n", CASES, ids=[f"{d}-{m}x{n}" for d, m, n in CASES])
def test_largest_accepted_sizes(dts, m, n, op):
    dt = np.float32 if dts == "f32" else np.float64
    print(f"limits {op} {dts} {m}x{n}: drawing inputs", flush=True)
    ins = make_inputs(op, m, n, dt, seed=31)
    print(f"limits {op} {dts} {m}x{n}: GPU", flush=True)
    got = gpu_outputs(op, ins, dt)
    print(f"limits {op} {dts} {m}x{n}: oracle", flush=True)
    ref = oracle_outputs(op, ins, dt)
    del ins
    for k, r in ref.items():
        assert got[k].shape == r.shape, f"{op} {k}: shape {got[k].shape} vs {r.shape}"
        err = normwise_sliced(got[k], r)
        print(f"limits {op} {dts} {m}x{n} {k}: normwise {err:.3e}", flush=True)
        assert err <= TOL[dt], f"{op} {dts} {m}x{n} {k}: normwise error {err:.3e} > {TOL[dt]:.0e}"
