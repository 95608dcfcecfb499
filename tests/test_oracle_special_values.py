"""The oracle on NaN and infinities, against brute force (CPU only).

The GPU special-value tests take the oracle's output classes (finite, +inf,
-inf, NaN) as the truth, so the oracle is pinned here on its own: every
operation on tiny inputs holding one NaN or infinity (in two cases beside an
exact zero), against the definitions written as plain Python loops over
Python floats, which follow IEEE double arithmetic (0 * inf is NaN, inf -
inf is NaN).  Outputs must agree in class at every position and, where
finite, to within rounding.
"""
import math

import numpy as np
import pytest

import oracle

ALPHA, BETA = 1.5, -0.75


def _rows(A):
    return [[float(v) for v in row] for row in A]


def _vec(v):
    return [float(e) for e in v]


def bf_matvec(A, x):
    return [sum(a * b for a, b in zip(row, x)) for row in A]


def bf_matvec_t(A, w):
    n = len(A[0])
    return [sum(A[i][j] * w[i] for i in range(len(A))) for j in range(n)]


def bf_gemver(A, u1, v1, u2, v2, y, z):
    m, n = len(A), len(A[0])
    Ahat = [[(A[i][j] + u1[i] * v1[j]) + u2[i] * v2[j] for j in range(n)] for i in range(m)]
    x = [BETA * sum(Ahat[i][j] * y[i] for i in range(m)) + z[j] for j in range(n)]
    w = [ALPHA * sum(Ahat[i][j] * x[j] for j in range(n)) for i in range(m)]
    return Ahat, x, w


def _cls(v):
    return 3 if math.isnan(v) else (1 if v == math.inf else (2 if v == -math.inf else 0))


def _same(got, want, what):
    got = np.asarray(got, np.float64).ravel()
    want = np.asarray(want, np.float64).ravel()
    assert got.shape == want.shape, what
    for k, (g, w) in enumerate(zip(got, want)):
        assert _cls(g) == _cls(w), f"{what}[{k}]: {g} vs {w}"
        if _cls(w) == 0:
            assert abs(g - w) <= 1e-12 * max(1.0, abs(w)), f"{what}[{k}]: {g} vs {w}"


def _inputs(seed, m, n):
    rng = np.random.default_rng(seed)
    draw = lambda *shape: rng.uniform(-1.0, 1.0, shape)
    return {"A": draw(m, n), "B": draw(m, n), "x": draw(n), "w": draw(m), "u1": draw(m), "v1": draw(n),
            "u2": draw(m), "v2": draw(n), "y": draw(m), "z": draw(n)}


# lists of (operand, position, value); positions are taken modulo the
# operand's shape.  The last two put an exact zero beside an infinity, so an
# oracle that skipped zero terms (instead of forming 0 * inf = NaN) fails.
CASES = [[("A", (1, 2), math.nan)], [("A", (0, 0), math.inf)], [("A", (2, 3), -math.inf)],
         [("B", (1, 1), math.inf)], [("x", 3, math.inf)], [("x", 0, math.nan)], [("w", 1, -math.inf)],
         [("u1", 2, math.inf)], [("v1", 1, -math.inf)], [("y", 0, math.inf)], [("z", 2, math.nan)],
         [("A", (1, 1), 0.0), ("x", 1, math.inf)], [("A", (0, 0), 0.0), ("w", 0, math.inf)]]


def _case_id(case):
    return "+".join(f"{k}-{'zero' if v == 0 else v}" for k, _, v in case)


@pytest.mark.parametrize("shape", [(3, 4), (1, 5), (4, 1)], ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("case", CASES, ids=_case_id)
def test_oracle_special_values_against_brute_force(case, shape):
    m, n = shape
    ins = _inputs(7 + m + n, m, n)
    for key, pos, value in case:
        arr = ins[key]
        if arr.ndim == 2:
            arr[pos[0] % m, pos[1] % n] = value
        else:
            arr[pos % arr.shape[0]] = value
    A, B = _rows(ins["A"]), _rows(ins["B"])
    x, w = _vec(ins["x"]), _vec(ins["w"])
    _same(oracle.matvec(ins["A"], ins["x"]), bf_matvec(A, x), "matvec")
    _same(oracle.matvec_t(ins["A"], ins["w"]), bf_matvec_t(A, w), "matvec_t")
    q, s = oracle.bicg(ins["A"], ins["x"], ins["w"])
    _same(q, bf_matvec(A, x), "bicg q")
    _same(s, bf_matvec_t(A, w), "bicg s")
    y, t = oracle.ata_x(ins["A"], ins["x"])
    t_bf = bf_matvec(A, x)
    _same(t, t_bf, "ata_x t")
    _same(y, bf_matvec_t(A, t_bf), "ata_x y")
    ax, bx = bf_matvec(A, x), bf_matvec(B, x)
    _same(oracle.axpby_mv(ALPHA, ins["A"], BETA, ins["B"], ins["x"]),
          [ALPHA * a + BETA * b for a, b in zip(ax, bx)], "axpby_mv")
    Ahat, gx, gw = oracle.gemver(ALPHA, BETA, ins["A"], ins["u1"], ins["v1"], ins["u2"], ins["v2"], ins["y"],
                                 ins["z"])
    bA, bx2, bw = bf_gemver(A, _vec(ins["u1"]), _vec(ins["v1"]), _vec(ins["u2"]), _vec(ins["v2"]),
                            _vec(ins["y"]), _vec(ins["z"]))
    _same(Ahat, bA, "gemver Ahat")
    _same(gx, bx2, "gemver x")
    _same(gw, bw, "gemver w")


@pytest.mark.parametrize("values", [[1.0, math.inf, 2.0], [math.inf, -1.0, -math.inf], [0.5, math.nan, math.inf],
                                    [-math.inf, -math.inf, 3.0]], ids=["inf", "inf-neg-inf", "nan", "neg-inf-twice"])
def test_oracle_sum_and_add_special_values(values):
    x = np.array(values)
    _same([oracle.reduce_sum(x)], [sum(values)], "reduce_sum")
    b = np.array([math.inf, -math.inf, 1.0])
    _same(oracle.vector_add(x, b), [p + q for p, q in zip(values, [math.inf, -math.inf, 1.0])], "vector_add")
