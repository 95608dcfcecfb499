"""The largest sizes the library accepts, on the GPU against the oracle.

- Rows of 65535 * 8192 elements, the longest accepted, as one-row matrices
  (2 GiB fp32, 4 GiB fp64).  The plans cut them into up to 65535 column
  panels, as many as one launch holds (the element-wise path, taken by the
  fp32 row of 65535 * 8192 - 1 elements, and fp64 GESUMMV), and the column
  outputs (A^T w, BICG's s, ATAX's y, GEMVER's x) are wider than one launch
  of the column reduce covers.
- 2^30 rows of one element, the most rows accepted (4 GiB fp32).
- The sum and the element-wise add over the longest accepted vector.

Every op runs on each; inputs come from the seeded generator, and every
output is compared in full with the oracle's by the normwise metric, in
slices so that no fp64 temporary of a whole output is formed.
"""
import numpy as np
import pytest

import oracle
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


VECTOR_CASES = [("f32", MAX_N - 1), ("f64", MAX_N)]


@pytest.mark.parametrize("dts,n", VECTOR_CASES, ids=[f"{d}-{n}" for d, n in VECTOR_CASES])
def test_vector_samples_at_the_longest_length(dts, n):
    """The sum (non-negative terms, held to the summation-depth bound and the
    product tolerance) and the element-wise add (bit-exact, every candidate)
    over the longest accepted vector; the fp32 length leaves a ragged tail
    after the last 16-byte vector."""
    import torch

    from paper_2512_22147_amd import datagen, mep
    from tests.sum_bound import sum_error_bound

    dt = np.float32 if dts == "f32" else np.float64
    print(f"limits vector samples {dts} n={n}: drawing inputs", flush=True)
    a = datagen.uniform(33, 0, (n,), dt)
    np.abs(a, out=a)
    ad = torch.from_numpy(a).to("cuda:0")
    got = float(mep.mep_reduce_sum(ad).cpu()[0])
    ref = oracle.reduce_sum(a)
    err = abs(got - ref) / abs(ref)
    print(f"limits reduce_sum {dts} n={n}: relative error {err:.3e}", flush=True)
    assert err <= min(TOL[dt], sum_error_bound(n, dt)), err
    b = datagen.normal(33, 1, (n,), dt)
    bd = torch.from_numpy(b).to("cuda:0")
    want = oracle.vector_add(a, b).astype(dt)
    del b
    code = mep.MEP_F32 if dt == np.float32 else mep.MEP_F64
    try:
        for v in range(mep.mep_variant_count(mep.MEP_OP_VECTOR_ADD, code, 1, n)):
            mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, v)
            c = mep.mep_vector_add(ad, bd)
            torch.cuda.synchronize()
            same = np.array_equal(c.cpu().numpy(), want)
            print(f"limits vector_add {dts} n={n} candidate {v}: bit-exact {same}", flush=True)
            assert same, f"candidate {v}"
            del c
    finally:
        mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, -1)
