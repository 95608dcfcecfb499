"""The vector samples of Table 3 ("reduction", "vectoradd") on the GPU,
through the C-ABI, against the CPU oracle.

Sum: |s - sum x| <= gamma_d * sum |x_i|, the worst-case error of any
summation whose longest chain of additions is d (tests/sum_bound.py derives
d from the kernel's summation depth); on non-negative inputs the sum does not
cancel, so the relative error |s - ref| / |ref| is held to that bound and to
the 1e-4 / 1e-12 tolerance of the products, which an all-zero result or one
missing workgroup partial both exceed.  Bit-exact on integer inputs.
Vector add: one correctly rounded addition per element, so bit-exact.
"""
import numpy as np
import pytest

import oracle

from tests.sum_bound import sum_error_bound

pytestmark = pytest.mark.gpu

TOL = {np.float32: 1e-4, np.float64: 1e-12}
SIZES = [0, 1, 3, 4, 17, 1000, 4099, (1 << 20) + 3, 1 << 26]


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_22147_amd import mep

    mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, -1)
    yield
    mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, -1)


def _dev(a, offset=0):
    """Copy a host array to the GPU, optionally `offset` elements past a
    16-byte boundary (the element-wise path)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a))
    raw = torch.empty(a.size + offset, dtype=t.dtype, device="cuda:0")
    d = raw[offset:]
    d.copy_(t)
    return d


@pytest.mark.parametrize("sign", ["mixed", "nonneg"])
@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("offset", [0, 1], ids=["aligned", "offset"])
def test_reduce_sum(n, dt, offset, sign):
    import torch

    from paper_2512_22147_amd import datagen, mep

    x = datagen.uniform(900 + n % 97, 0, (n,), dt)
    if sign == "nonneg":
        x = np.abs(x)
    ref = oracle.reduce_sum(x)
    scale = float(np.abs(x.astype(np.float64)).sum())
    xd = _dev(x, offset)
    s1 = mep.mep_reduce_sum(xd)
    s2 = mep.mep_reduce_sum(xd)
    torch.cuda.synchronize()
    got = float(s1.cpu()[0])
    assert abs(got - ref) <= sum_error_bound(n, dt, offset=offset) * scale, (got, ref, scale)
    if sign == "nonneg" and n > 0:
        assert abs(got - ref) / abs(ref) <= TOL[dt], (got, ref)
    assert s1.cpu().numpy().tobytes() == s2.cpu().numpy().tobytes(), "not reproducible"


@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
def test_reduce_sum_integer_exact(dt):
    import torch

    from paper_2512_22147_amd import datagen, mep

    n = (1 << 22) + 5
    x = datagen.ternary(911, 0, (n,), dt)
    got = mep.mep_reduce_sum(_dev(x))
    torch.cuda.synchronize()
    assert float(got.cpu()[0]) == oracle.reduce_sum(x) == float(x.astype(np.int64).sum())


@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("offset", [0, 1], ids=["aligned", "offset"])
def test_vector_add_bit_exact(n, dt, offset):
    import torch

    from paper_2512_22147_amd import datagen, mep

    a = datagen.uniform(920 + n % 89, 0, (n,), dt)
    b = datagen.normal(920 + n % 89, 1, (n,), dt)
    ref = oracle.vector_add(a, b).astype(dt)
    guard = 4096
    ad, bd = _dev(a, offset), _dev(b, offset)
    count = mep.mep_variant_count(mep.MEP_OP_VECTOR_ADD, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, 1, n)
    assert count >= 2
    for v in range(count):
        mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, v)
        c_all = torch.full((n + guard,), 777.0, dtype=torch.float32 if dt == np.float32 else torch.float64,
                           device="cuda:0")
        c = mep.mep_vector_add(ad, bd, c=c_all[:n])
        torch.cuda.synchronize()
        assert np.array_equal(c.cpu().numpy(), ref), f"candidate {v}"
        assert bool((c_all[n:] == 777.0).all()), f"candidate {v} wrote past c"


@pytest.mark.parametrize("name", ["reduce_sum_256m", "vector_add_256m"])
def test_vector_workloads_full_size(name):
    """The benchmark sizes (2^28 fp32 elements) in the launch configuration
    bench.py times."""
    import torch

    from paper_2512_22147_amd import datagen, mep

    ins = datagen.make_inputs(name)
    if name == "reduce_sum_256m":
        # non-negative terms: the relative error is meaningful (an all-zero
        # result or a missing workgroup partial fails; tests/test_sum_bound.py
        # shows both on these inputs)
        x = ins["x"]
        assert float(x.min()) >= 0.0
        got = mep.mep_reduce_sum(_dev(x))
        torch.cuda.synchronize()
        ref = oracle.reduce_sum(x)
        err = abs(float(got.cpu()[0]) - ref) / abs(ref)
        assert err <= min(1e-4, sum_error_bound(x.size, np.float32)), err
    else:
        ref = oracle.vector_add(ins["a"], ins["b"]).astype(np.float32)
        ad, bd = _dev(ins["a"]), _dev(ins["b"])
        for v in range(mep.mep_variant_count(mep.MEP_OP_VECTOR_ADD, mep.MEP_F32, 1, ad.numel())):
            mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, v)
            c = mep.mep_vector_add(ad, bd)
            torch.cuda.synchronize()
            assert np.array_equal(c.cpu().numpy(), ref), f"candidate {v}"
