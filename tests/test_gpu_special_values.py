"""IEEE special values through every operation and every candidate shape.

One NaN or infinity is placed in A (the matrix's last element, or the first
element of a middle row), in the vector operand multiplied into A (its last
element), or in another operand (BICG's r, GESUMMV's B, GEMVER's u1, y, z),
on shapes that take the row-group path, the element-wise path for
misaligned rows, the narrow-row path and column panels.  With a single
special value per input and no finite partial sum near overflow, whether an
output is NaN, +inf, -inf or finite does not depend on the order of
summation nor on the precision, so every candidate must match the oracle's
class at every position, and every finite output must match it within the
normwise tolerance.  A kernel that reads past a row's end and cancels the
extra elements with zero weights (0 * inf is NaN), or that lets a padding
lane or a column partial carry a value into another output, fails here.
"""
import numpy as np
import pytest

from tests.gpu_cases import OPS, TOL, gpu_outputs, make_inputs, op_code, oracle_outputs

pytestmark = pytest.mark.gpu

# row groups, misaligned rows (element-wise), narrow rows, column panels, one
# row, where an infinity in the vector gives definite infinities in ATAX's y
# and GEMVER's x that a padding row of the last block would turn into NaN,
# a streamed matrix (past 128 MiB: non-temporal shapes, which skip the rows
# past the end instead of zeroing them), and a streamed one in column panels
# (with the cyclic, rotated and blocked row maps among its candidates)
SHAPES = [(1037, 2052), (1001, 2051), (1001, 8), (3, 40001), (1, 4100), (2051, 16384), (1025, 40000)]

# the vector operand multiplied into A, with its length
VECTOR_IN = {"matvec": ("x", 1), "matvec_t": ("w", 0), "bicg": ("x", 1), "ata_x": ("x", 1),
             "axpby_mv": ("x", 1), "gemver": ("v1", 1)}


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_22147_amd import mep

    for op in range(8):
        mep.mep_set_variant(op, -1)
    yield
    for op in range(8):
        mep.mep_set_variant(op, -1)


def _classes(a):
    a = np.asarray(a, np.float64).ravel()
    return np.where(np.isnan(a), 3, np.where(np.isposinf(a), 1, np.where(np.isneginf(a), 2, 0)))


def _inject(op, ins, where):
    m, n = ins["A"].shape
    if where == "nan-last-element":
        ins["A"][m - 1, n - 1] = np.nan
    elif where == "inf-row-start":
        ins["A"][m // 2, 0] = np.inf
    else:
        key, axis = VECTOR_IN[op]
        ins[key][(m, n)[axis] - 1] = -np.inf


def _check_every_candidate(op, ins, dt):
    """The default and every candidate against the oracle: same class at
    every output position, finite outputs within the normwise tolerance."""
    import torch

    from paper_2512_22147_amd import mep

    m, n = ins["A"].shape
    ref = oracle_outputs(op, ins, dt)
    want = {k: _classes(r) for k, r in ref.items()}
    assert any((c != 0).any() for c in want.values()), "the special value reached no output"
    code = op_code(op)
    count = mep.mep_variant_count(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n)
    # the inputs go to the GPU once; no operation writes them
    dins = {k: torch.from_numpy(np.ascontiguousarray(v)).to("cuda:0") for k, v in ins.items()}
    for v in [-1] + list(range(count)):
        mep.mep_set_variant(code, v)
        got = gpu_outputs(op, dins, dt)
        for k, r in ref.items():
            g = np.asarray(got[k], np.float64).ravel()
            r = np.asarray(r, np.float64).ravel()
            bad = np.flatnonzero(_classes(g) != want[k])
            assert bad.size == 0, (f"{op} {k} candidate {v}: {bad.size} outputs differ in class from the "
                                   f"oracle, first at {bad[0]}: {g[bad[0]]} vs {r[bad[0]]}")
            fin = want[k] == 0
            if fin.any():
                scale = float(np.max(np.abs(r[fin])))
                err = float(np.max(np.abs(g[fin] - r[fin])))
                err = err / scale if scale > 0 else err
                assert err <= TOL[dt], f"{op} {k} candidate {v}: finite outputs differ by {err:.3e}"


@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("where", ["nan-last-element", "inf-row-start", "neg-inf-vector-last"])
def test_special_values_every_candidate(where, shape, op, dt):
    m, n = shape
    ins = make_inputs(op, m, n, dt, seed=88 + m + n)
    _inject(op, ins, where)
    _check_every_candidate(op, ins, dt)


# the other operands: BICG's r, GESUMMV's B, GEMVER's u1, y and z (operand,
# position as a function of the shape, value)
SECOND = [("bicg", "w", lambda m, n: m - 1, np.inf), ("bicg", "w", lambda m, n: 0, np.nan),
          ("axpby_mv", "B", lambda m, n: (m // 2, 0), np.nan),
          ("axpby_mv", "B", lambda m, n: (m - 1, n - 1), -np.inf),
          ("gemver", "u1", lambda m, n: m - 1, np.inf), ("gemver", "y", lambda m, n: m - 1, -np.inf),
          ("gemver", "z", lambda m, n: n - 1, np.nan)]


@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("case", range(len(SECOND)),
                         ids=[f"{o}-{k}-{v}" for o, k, _, v in SECOND])
def test_special_values_in_other_operands(case, shape, dt):
    op, key, pos, value = SECOND[case]
    m, n = shape
    ins = make_inputs(op, m, n, dt, seed=77 + m + n)
    ins[key][pos(m, n)] = value
    _check_every_candidate(op, ins, dt)


def _sum_class(x):
    return int(_classes(np.array([x]))[0])


@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
@pytest.mark.parametrize("n", [5, 4099, (1 << 20) + 3])
@pytest.mark.parametrize("offset", [0, 1], ids=["aligned", "offset"])
@pytest.mark.parametrize("case", ["inf", "inf-and-neg-inf", "nan"])
def test_vector_samples_special_values(case, offset, n, dt):
    """The sum is +inf (one infinity) or NaN (infinities of both signs, or a NaN)
    in any order of summation; the add is one
    IEEE addition per element (inf + -inf is NaN), compared value for value
    with NaN equal to NaN, under every candidate; padding lanes add nothing."""
    import torch

    import oracle
    from paper_2512_22147_amd import datagen, mep

    tdt = torch.float32 if dt == np.float32 else torch.float64
    code = mep.MEP_F32 if dt == np.float32 else mep.MEP_F64
    x = datagen.uniform(61 + n, 0, (n,), dt)
    y = datagen.uniform(61 + n, 1, (n,), dt)
    x[n - 1] = np.inf
    if case == "inf-and-neg-inf":
        x[n // 2] = -np.inf
        y[n // 2] = np.inf  # the add: -inf + inf at one position
    elif case == "nan":
        x[0] = np.nan
        y[n - 1] = -np.inf  # the add: inf + -inf at the last position
    want = _sum_class(oracle.reduce_sum(x))
    assert want == {"inf": 1, "inf-and-neg-inf": 3, "nan": 3}[case]

    def dev(a):
        raw = torch.empty(n + offset, dtype=tdt, device="cuda:0")
        raw[offset:].copy_(torch.from_numpy(a))
        return raw[offset:]

    xd, yd = dev(x), dev(y)
    for v in [-1] + list(range(mep.mep_variant_count(mep.MEP_OP_REDUCE_SUM, code, 1, n))):
        mep.mep_set_variant(mep.MEP_OP_REDUCE_SUM, v)
        got = float(mep.mep_reduce_sum(xd).cpu()[0])
        assert _sum_class(got) == want, f"sum candidate {v}: {got}"
    mep.mep_set_variant(mep.MEP_OP_REDUCE_SUM, -1)
    ref = oracle.vector_add(x, y).astype(dt)
    for v in [-1] + list(range(mep.mep_variant_count(mep.MEP_OP_VECTOR_ADD, code, 1, n))):
        mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, v)
        c = mep.mep_vector_add(xd, yd)
        torch.cuda.synchronize()
        assert np.array_equal(c.cpu().numpy(), ref, equal_nan=True), f"add candidate {v}"
    mep.mep_set_variant(mep.MEP_OP_VECTOR_ADD, -1)
