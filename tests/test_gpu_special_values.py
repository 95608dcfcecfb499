"""IEEE special values through every operation and every candidate shape.

One NaN or infinity is placed in A (the matrix's last element, or the first
element of a middle row) or in the vector operand multiplied into A (its last
element), on shapes that take the row-group path, the element-wise path for
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

# row groups, misaligned rows (element-wise), narrow rows, column panels, and
# one row, where an infinity in the vector gives definite infinities in
# ATAX's y and GEMVER's x that a padding row of the last block would turn
# into NaN
SHAPES = [(1037, 2052), (1001, 2051), (1001, 8), (3, 40001), (1, 4100)]

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


@pytest.mark.parametrize("dt", [np.float32, np.float64], ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("where", ["nan-last-element", "inf-row-start", "neg-inf-vector-last"])
def test_special_values_every_candidate(where, shape, op, dt):
    from paper_2512_22147_amd import mep

    m, n = shape
    ins = make_inputs(op, m, n, dt, seed=88 + m + n)
    _inject(op, ins, where)
    ref = oracle_outputs(op, ins, dt)
    want = {k: _classes(r) for k, r in ref.items()}
    assert any((c != 0).any() for c in want.values()), "the special value reached no output"
    code = op_code(op)
    count = mep.mep_variant_count(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n)
    for v in [-1] + list(range(count)):
        mep.mep_set_variant(code, v)
        got = gpu_outputs(op, ins, dt)
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
