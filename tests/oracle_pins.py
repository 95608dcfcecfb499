"""Pins for the CPU oracle: checks against what mathematics fixes, never
against the oracle itself.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError on a
mismatch.  They are run against the real oracle (``test_oracle_pins.py``) and
against copies of it with planted mistakes (``test_oracle_mutants.py``), which
must each fail at least one pin.

What pins the oracle:
* exact rational arithmetic (``fractions.Fraction``) on tiny inputs, with the
  fp64 dot-product error bound |fl(a.b) - a.b| <= gamma_k |a|.|b|,
  gamma_k = k u / (1 - k u), u = 2^-53 (Higham, Accuracy and Stability of
  Numerical Algorithms, 2nd ed., Sec. 3.1);
* the identity A^T (A x) = (A^T A) x with A^T A formed exactly;
* the adjoint identity w.(A x) = (A^T w).x;
* closed forms for A = I, A = all-ones, A = diag(d), B = A;
* integer-valued inputs, whose products and sums are exact in fp64, compared
  bit for bit with numpy's int64 matrix product;
* numpy's float64 ``@`` as an independent library routine;
* on NaN and infinities, the definitions as plain Python loops over Python
  floats, which follow IEEE double arithmetic (0 * inf is NaN).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from paper_2512_22147_amd import datagen

U64 = Fraction(1, 2**53)


def gamma(k: int) -> Fraction:
    return k * U64 / (1 - k * U64)


def F(v) -> Fraction:
    return Fraction(float(v))


def exact_matvec(A, x):
    m, n = A.shape
    return [sum((F(A[i, j]) * F(x[j]) for j in range(n)), Fraction(0)) for i in range(m)]


def exact_matvec_t(A, w):
    m, n = A.shape
    return [sum((F(A[i, j]) * F(w[i]) for i in range(m)), Fraction(0)) for j in range(n)]


def abs_matvec(A, x):
    m, n = A.shape
    return [sum((abs(F(A[i, j]) * F(x[j])) for j in range(n)), Fraction(0)) for i in range(m)]


def abs_matvec_t(A, w):
    m, n = A.shape
    return [sum((abs(F(A[i, j]) * F(w[i])) for i in range(m)), Fraction(0)) for j in range(n)]


def _within(got, exact, bound, what):
    assert len(got) == len(exact) == len(bound), what
    for i, (g, e, b) in enumerate(zip(got, exact, bound)):
        gv = float(g)
        assert np.isfinite(gv), f"{what}[{i}] not finite"
        err = abs(F(gv) - e)
        assert err <= b, f"{what}[{i}]: |{gv!r} - exact| = {float(err):.3e} > bound {float(b):.3e}"


SMALL_SHAPES = [(1, 1), (1, 8), (8, 1), (8, 8), (5, 7), (7, 5), (3, 16)]


def _small_inputs(m, n, seed, dtype):
    A = datagen.uniform(seed, 0, (m, n), dtype)
    x = datagen.uniform(seed, 1, (n,), dtype)
    w = datagen.uniform(seed, 2, (m,), dtype)
    B = datagen.uniform(seed, 3, (m, n), dtype)
    return A, x, w, B


def pin_bruteforce_matvec(orc):
    for dt in (np.float32, np.float64):
        for s, (m, n) in enumerate(SMALL_SHAPES):
            A, x, _, _ = _small_inputs(m, n, 100 + s, dt)
            y = orc.matvec(A, x)
            _within(y, exact_matvec(A, x), [gamma(n) * b for b in abs_matvec(A, x)],
                    f"matvec {m}x{n} {np.dtype(dt).name}")


def pin_bruteforce_matvec_t(orc):
    for dt in (np.float32, np.float64):
        for s, (m, n) in enumerate(SMALL_SHAPES):
            A, _, w, _ = _small_inputs(m, n, 200 + s, dt)
            z = orc.matvec_t(A, w)
            _within(z, exact_matvec_t(A, w), [gamma(m) * b for b in abs_matvec_t(A, w)],
                    f"matvec_t {m}x{n} {np.dtype(dt).name}")


def _ata_bound(A, x, m, n):
    # |y^ - A^T A x| <= gamma_m |A|^T |t^| + |A|^T |t^ - t|
    #              <= (gamma_m (1 + gamma_n) + gamma_n) |A|^T |A| |x|
    ax = abs_matvec(A, x)
    aat = [sum((abs(F(A[i, j])) * ax[i] for i in range(m)), Fraction(0)) for j in range(n)]
    g = gamma(m) * (1 + gamma(n)) + gamma(n)
    return [g * v for v in aat]


def pin_bruteforce_ata_x(orc):
    for dt in (np.float32, np.float64):
        for s, (m, n) in enumerate(SMALL_SHAPES):
            A, x, _, _ = _small_inputs(m, n, 300 + s, dt)
            y, t = orc.ata_x(A, x)
            _within(t, exact_matvec(A, x), [gamma(n) * b for b in abs_matvec(A, x)],
                    f"ata_x t {m}x{n}")
            exact_t = exact_matvec(A, x)
            exact_y = [sum((F(A[i, j]) * exact_t[i] for i in range(m)), Fraction(0))
                       for j in range(n)]
            _within(y, exact_y, _ata_bound(A, x, m, n), f"ata_x y {m}x{n}")


def pin_bruteforce_bicg(orc):
    for s, (m, n) in enumerate(SMALL_SHAPES):
        A, p, r, _ = _small_inputs(m, n, 400 + s, np.float32)
        q, sv = orc.bicg(A, p, r)
        _within(q, exact_matvec(A, p), [gamma(n) * b for b in abs_matvec(A, p)], "bicg q")
        _within(sv, exact_matvec_t(A, r), [gamma(m) * b for b in abs_matvec_t(A, r)], "bicg s")


def pin_bruteforce_axpby(orc):
    for s, (m, n) in enumerate(SMALL_SHAPES):
        A, x, _, B = _small_inputs(m, n, 500 + s, np.float32)
        alpha, beta = float(np.float32(1.5)), float(np.float32(1.2))
        y = orc.axpby_mv(alpha, A, beta, B, x)
        ea, eb = exact_matvec(A, x), exact_matvec(B, x)
        aa, ab = abs_matvec(A, x), abs_matvec(B, x)
        a_, b_ = F(alpha), F(beta)
        exact = [a_ * u + b_ * v for u, v in zip(ea, eb)]
        # dot products carry gamma_n, each product and the sum one more u
        g = gamma(n + 2)
        bound = [g * (abs(a_) * u + abs(b_) * v) for u, v in zip(aa, ab)]
        _within(y, exact, bound, f"axpby {m}x{n}")


def pin_identity_ata(orc):
    """A^T (A x) equals (A^T A) x with A^T A formed exactly."""
    for (m, n, seed) in ((12, 16, 7), (16, 12, 8), (16, 16, 9)):
        A = datagen.uniform(seed, 0, (m, n), np.float32)
        x = datagen.uniform(seed, 1, (n,), np.float32)
        AtA = [[sum((F(A[i, j]) * F(A[i, k]) for i in range(m)), Fraction(0))
                for k in range(n)] for j in range(n)]
        exact = [sum((AtA[j][k] * F(x[k]) for k in range(n)), Fraction(0)) for j in range(n)]
        y, _ = orc.ata_x(A, x)
        _within(y, exact, _ata_bound(A, x, m, n), f"A^T A identity {m}x{n}")


def pin_adjoint(orc):
    """w.(A x) = (A^T w).x up to the two products' error bounds."""
    for (m, n, seed) in ((33, 47, 21), (47, 33, 22)):
        A = datagen.uniform(seed, 0, (m, n), np.float64)
        x = datagen.uniform(seed, 1, (n,), np.float64)
        w = datagen.uniform(seed, 2, (m,), np.float64)
        y = orc.matvec(A, x)
        z = orc.matvec_t(A, w)
        lhs = sum((F(w[i]) * F(y[i]) for i in range(m)), Fraction(0))
        rhs = sum((F(z[j]) * F(x[j]) for j in range(n)), Fraction(0))
        ax = abs_matvec(A, x)
        scale = sum((abs(F(w[i])) * ax[i] for i in range(m)), Fraction(0))
        assert abs(lhs - rhs) <= (gamma(n) + gamma(m)) * scale, "adjoint identity"
        # ATAX: x.(A^T A x) = |A x|^2 >= 0
        ya, t = orc.ata_x(A, x)
        xy = sum((F(x[j]) * F(ya[j]) for j in range(n)), Fraction(0))
        tt = sum((F(v) * F(v) for v in t), Fraction(0))
        assert abs(xy - tt) <= 4 * (gamma(n) + gamma(m)) * scale_sq(A, x), "x.y = |Ax|^2"
        assert xy > 0


def scale_sq(A, x):
    ax = abs_matvec(A, x)
    return sum((v * v for v in ax), Fraction(0))


def pin_closed_forms(orc):
    n = 37
    x = datagen.uniform(31, 1, (n,), np.float32)
    w = datagen.uniform(31, 2, (n,), np.float32)
    eye = np.eye(n, dtype=np.float32)
    assert np.array_equal(orc.matvec(eye, x), x.astype(np.float64)), "I x = x"
    assert np.array_equal(orc.matvec_t(eye, w), w.astype(np.float64)), "I^T w = w"
    y, t = orc.ata_x(eye, x)
    assert np.array_equal(y, x.astype(np.float64)) and np.array_equal(t, x.astype(np.float64)), \
        "I^T I x = x"
    # alpha = 1.5, beta = 0.25 are dyadic, so (alpha + beta) x is exact
    assert np.array_equal(orc.axpby_mv(1.5, eye, 0.25, eye, x), 1.75 * x.astype(np.float64)), \
        "GESUMMV with A = B = I"
    q, s = orc.bicg(eye, x, w)
    assert np.array_equal(q, x.astype(np.float64)) and np.array_equal(s, w.astype(np.float64))

    # all-ones m x n: sums of fp32 values in [-1, 1) are exact in fp64 here
    m, n2 = 33, 65
    ones = np.ones((m, n2), dtype=np.float32)
    x2 = datagen.uniform(32, 1, (n2,), np.float32)
    w2 = datagen.uniform(32, 2, (m,), np.float32)
    sx = float(sum(F(v) for v in x2))
    sw = float(sum(F(v) for v in w2))
    assert np.array_equal(orc.matvec(ones, x2), np.full(m, sx)), "ones x"
    assert np.array_equal(orc.matvec_t(ones, w2), np.full(n2, sw)), "ones^T w"
    ya, ta = orc.ata_x(ones, x2)
    assert np.array_equal(ta, np.full(m, sx)) and np.array_equal(ya, np.full(n2, m * sx)), \
        "ones^T ones x = m (sum x) 1"

    # diag(d): products of two fp32 values are exact in fp64
    d = datagen.uniform(33, 0, (n,), np.float32)
    D = np.diag(d).astype(np.float32)
    assert np.array_equal(orc.matvec(D, x), d.astype(np.float64) * x.astype(np.float64))
    assert np.array_equal(orc.matvec_t(D, w), d.astype(np.float64) * w.astype(np.float64))
    yd, _ = orc.ata_x(D, x)
    dd = d.astype(np.float64)
    assert np.array_equal(yd, dd * (dd * x.astype(np.float64))), "diag ATAX"

    # B = A: alpha A x + beta A x = (alpha + beta) A x, exact on integer inputs
    At = datagen.ternary(34, 0, (29, 41), np.float32)
    xt = datagen.ternary(34, 1, (41,), np.float32)
    ref = 1.75 * (At.astype(np.int64) @ xt.astype(np.int64)).astype(np.float64)
    assert np.array_equal(orc.axpby_mv(1.5, At, 0.25, At, xt), ref), "B = A"


def pin_integer_exact(orc):
    """Ternary inputs: every partial sum is a small integer, so the fp64
    result must equal numpy's int64 product bit for bit."""
    for (m, n, seed) in ((300, 500, 41), (500, 300, 42), (1, 700, 43), (700, 1, 44)):
        A = datagen.ternary(seed, 0, (m, n), np.float32)
        x = datagen.ternary(seed, 1, (n,), np.float32)
        w = datagen.ternary(seed, 2, (m,), np.float32)
        B = datagen.ternary(seed, 3, (m, n), np.float32)
        Ai, xi, wi, Bi = (a.astype(np.int64) for a in (A, x, w, B))
        assert np.array_equal(orc.matvec(A, x), (Ai @ xi).astype(np.float64)), "int matvec"
        assert np.array_equal(orc.matvec_t(A, w), (Ai.T @ wi).astype(np.float64)), "int matvec_t"
        y, t = orc.ata_x(A, x)
        assert np.array_equal(t, (Ai @ xi).astype(np.float64))
        assert np.array_equal(y, (Ai.T @ (Ai @ xi)).astype(np.float64)), "int ata_x"
        q, s = orc.bicg(A, x, w)
        assert np.array_equal(q, (Ai @ xi).astype(np.float64))
        assert np.array_equal(s, (Ai.T @ wi).astype(np.float64)), "int bicg"
        yy = orc.axpby_mv(1.5, A, 0.25, B, x)
        ref = 1.5 * (Ai @ xi).astype(np.float64) + 0.25 * (Bi @ xi).astype(np.float64)
        assert np.array_equal(yy, ref), "int axpby"


def _normwise(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


def pin_numpy_crosscheck(orc):
    """numpy float64 @ agrees to 1e-13 normwise (a library routine as an
    independent cross-check)."""
    for (m, n, seed) in ((257, 263, 51), (263, 257, 52), (1024, 64, 53)):
        A = datagen.uniform(seed, 0, (m, n), np.float64)
        x = datagen.uniform(seed, 1, (n,), np.float64)
        w = datagen.uniform(seed, 2, (m,), np.float64)
        B = datagen.normal(seed, 3, (m, n), np.float64)
        assert _normwise(orc.matvec(A, x), A @ x) <= 1e-13
        assert _normwise(orc.matvec_t(A, w), A.T @ w) <= 1e-13
        y, _ = orc.ata_x(A, x)
        assert _normwise(y, A.T @ (A @ x)) <= 1e-13
        q, s = orc.bicg(A, x, w)
        assert _normwise(q, A @ x) <= 1e-13 and _normwise(s, A.T @ w) <= 1e-13
        assert _normwise(orc.axpby_mv(1.5, A, 1.2, B, x), 1.5 * (A @ x) + 1.2 * (B @ x)) <= 1e-13


def pin_reduce_sum(orc):
    """Exact rational sums within the recursive-summation bound
    gamma_{n-1} sum |x_i|; integer inputs exactly; closed forms."""
    for n, seed in ((1, 71), (2, 72), (17, 73), (100, 74)):
        x = datagen.uniform(seed, 0, (n,), np.float64)
        exact = sum((F(v) for v in x), Fraction(0))
        bound = gamma(max(n - 1, 1)) * sum((abs(F(v)) for v in x), Fraction(0))
        assert abs(F(orc.reduce_sum(x)) - exact) <= bound, f"reduce_sum n={n}"
    t = datagen.ternary(75, 0, (100000,), np.float32)
    assert orc.reduce_sum(t) == float(t.astype(np.int64).sum()), "integer sum"
    assert orc.reduce_sum(np.ones(12345)) == 12345.0
    assert orc.reduce_sum(np.zeros(0)) == 0.0
    assert orc.reduce_sum(np.array([0.5, 0.25, -0.75])) == 0.0


def pin_vector_add(orc):
    """Each sum is one correctly rounded addition: exact for fp32 inputs in
    fp64, and equal to the exactly rounded rational sum for fp64 inputs."""
    a = datagen.uniform(81, 0, (1000,), np.float32)
    b = datagen.uniform(81, 1, (1000,), np.float32)
    c = orc.vector_add(a, b)
    assert all(F(ci) == F(ai) + F(bi) for ai, bi, ci in zip(a, b, c)), "fp32 sums exact in fp64"
    a = datagen.uniform(82, 0, (200,), np.float64)
    b = datagen.normal(82, 1, (200,), np.float64)
    c = orc.vector_add(a, b)
    for ai, bi, ci in zip(a, b, c):
        e = F(ai) + F(bi)
        assert abs(F(ci) - e) <= U64 * abs(e), "fp64 sum correctly rounded"
    assert np.array_equal(orc.vector_add(np.arange(5.0), -np.arange(5.0)), np.zeros(5))


def _gemver_inputs(m, n, seed, dt, draw=None):
    draw = draw or datagen.uniform
    return dict(A=draw(seed, 0, (m, n), dt), u1=draw(seed, 1, (m,), dt), v1=draw(seed, 2, (n,), dt),
                u2=draw(seed, 3, (m,), dt), v2=draw(seed, 4, (n,), dt), y=draw(seed, 5, (m,), dt),
                z=draw(seed, 6, (n,), dt))


def pin_gemver(orc):
    """Exact rational GEMVER on small shapes within first-order bounds;
    integer inputs bit for bit against int64 products; rank-1 closed form."""
    for (m, n, seed) in ((1, 1, 91), (3, 5, 92), (6, 4, 93), (8, 8, 94)):
        g = _gemver_inputs(m, n, seed, np.float32)
        al, be = F(1.5), F(np.float32(1.2))
        Ah, x, w = orc.gemver(1.5, float(np.float32(1.2)), **g)
        A = [[F(v) for v in row] for row in g["A"]]
        E = [[A[i][j] + F(g["u1"][i]) * F(g["v1"][j]) + F(g["u2"][i]) * F(g["v2"][j]) for j in range(n)]
             for i in range(m)]
        aE = [[abs(A[i][j]) + abs(F(g["u1"][i]) * F(g["v1"][j])) + abs(F(g["u2"][i]) * F(g["v2"][j]))
               for j in range(n)] for i in range(m)]
        for i in range(m):
            _within(Ah[i], E[i], [gamma(4) * v for v in aE[i]], f"gemver Ahat row {i}")
        ex = [be * sum((E[i][j] * F(g["y"][i]) for i in range(m)), Fraction(0)) + F(g["z"][j]) for j in range(n)]
        bx = [gamma(m + 6) * (abs(be) * sum((aE[i][j] * abs(F(g["y"][i])) for i in range(m)), Fraction(0))
                              + abs(F(g["z"][j]))) for j in range(n)]
        _within(x, ex, bx, "gemver x")
        # w uses the oracle's own x: check it against exact arithmetic on that x
        ew = [al * sum((E[i][j] * F(x[j]) for j in range(n)), Fraction(0)) for i in range(m)]
        bw = [gamma(n + 6) * abs(al) * sum((aE[i][j] * abs(F(x[j])) for j in range(n)), Fraction(0))
              for i in range(m)]
        _within(w, ew, bw, "gemver w")
    # integer inputs: every value exact in fp64
    g = _gemver_inputs(120, 90, 95, np.float32, datagen.ternary)
    Ah, x, w = orc.gemver(2.0, 3.0, **g)
    I = {k: v.astype(np.int64) for k, v in g.items()}
    Ei = I["A"] + np.outer(I["u1"], I["v1"]) + np.outer(I["u2"], I["v2"])
    xi = 3 * (Ei.T @ I["y"]) + I["z"]
    wi = 2 * (Ei @ xi)
    assert np.array_equal(Ah, Ei.astype(np.float64)) and np.array_equal(x, xi.astype(np.float64))
    assert np.array_equal(w, wi.astype(np.float64)), "integer gemver"
    # A = 0, u2 = 0: Ahat = u1 v1^T, x = beta (u1.y) v1 + z, w = alpha (v1.x) u1; dyadic values make it exact
    m, n = 7, 9
    u1 = np.arange(1, m + 1, dtype=np.float64) / 4
    v1 = np.arange(-4, n - 4, dtype=np.float64) / 2
    y = np.ones(m)
    z = np.full(n, 0.5)
    Ah, x, w = orc.gemver(0.5, 2.0, np.zeros((m, n)), u1, v1, np.zeros(m), np.zeros(n), y, z)
    assert np.array_equal(Ah, np.outer(u1, v1))
    assert np.array_equal(x, 2.0 * u1.sum() * v1 + z)
    assert np.array_equal(w, 0.5 * float(v1 @ x) * u1)


# --- NaN and infinities: brute force over Python floats ---------------------

SV_ALPHA, SV_BETA = 1.5, -0.75

# lists of (operand, position, value); positions are taken modulo the
# operand's shape.  The last four put an exact zero beside an infinity, so an
# oracle that skipped zero terms or zero weights (instead of forming
# 0 * inf = NaN) fails.
SV_CASES = [[("A", (1, 2), float("nan"))], [("A", (0, 0), float("inf"))], [("A", (2, 3), -float("inf"))],
            [("B", (1, 1), float("inf"))], [("x", 3, float("inf"))], [("x", 0, float("nan"))],
            [("w", 1, -float("inf"))], [("u1", 2, float("inf"))], [("v1", 1, -float("inf"))],
            [("y", 0, float("inf"))], [("z", 2, float("nan"))],
            [("A", (1, 1), 0.0), ("x", 1, float("inf"))], [("A", (0, 0), 0.0), ("w", 0, float("inf"))],
            [("A", (1, 2), float("inf")), ("w", 1, 0.0)], [("A", (2, 1), float("inf")), ("x", 1, 0.0)]]
SV_SHAPES = [(3, 4), (1, 5), (4, 1)]


def _sv_class(v):
    return 3 if v != v else (1 if v == float("inf") else (2 if v == -float("inf") else 0))


def _sv_same(got, want, what):
    got = np.asarray(got, np.float64).ravel()
    assert got.shape == (len(want),), what
    for k, (g, w) in enumerate(zip(got.tolist(), want)):
        assert _sv_class(g) == _sv_class(w), f"{what}[{k}]: {g} vs {w}"
        if _sv_class(w) == 0:
            assert abs(g - w) <= 1e-12 * max(1.0, abs(w)), f"{what}[{k}]: {g} vs {w}"


def _sv_inputs(case, m, n):
    rng = np.random.default_rng(7 + m + n)
    ins = {k: rng.uniform(-1.0, 1.0, shape) for k, shape in
           (("A", (m, n)), ("B", (m, n)), ("x", (n,)), ("w", (m,)), ("u1", (m,)), ("v1", (n,)), ("u2", (m,)),
            ("v2", (n,)), ("y", (m,)), ("z", (n,)))}
    for key, pos, value in case:
        if ins[key].ndim == 2:
            ins[key][pos[0] % m, pos[1] % n] = value
        else:
            ins[key][pos % ins[key].shape[0]] = value
    return ins


def special_values_case(orc, case, m, n):
    """Every operation of the oracle on one special-value case, against the
    definitions as loops over Python floats."""
    ins = _sv_inputs(case, m, n)
    A = [[float(v) for v in row] for row in ins["A"]]
    B = [[float(v) for v in row] for row in ins["B"]]
    x, w = [float(v) for v in ins["x"]], [float(v) for v in ins["w"]]
    u1, v1, u2, v2, yv, z = ([float(e) for e in ins[k]] for k in ("u1", "v1", "u2", "v2", "y", "z"))

    def mv(M, v):
        return [sum(a * b for a, b in zip(row, v)) for row in M]

    def mvt(M, v):
        return [sum(M[i][j] * v[i] for i in range(len(M))) for j in range(len(M[0]))]

    _sv_same(orc.matvec(ins["A"], ins["x"]), mv(A, x), "matvec")
    _sv_same(orc.matvec_t(ins["A"], ins["w"]), mvt(A, w), "matvec_t")
    q, s = orc.bicg(ins["A"], ins["x"], ins["w"])
    _sv_same(q, mv(A, x), "bicg q")
    _sv_same(s, mvt(A, w), "bicg s")
    y, t = orc.ata_x(ins["A"], ins["x"])
    _sv_same(t, mv(A, x), "ata_x t")
    _sv_same(y, mvt(A, mv(A, x)), "ata_x y")
    _sv_same(orc.axpby_mv(SV_ALPHA, ins["A"], SV_BETA, ins["B"], ins["x"]),
             [SV_ALPHA * a + SV_BETA * b for a, b in zip(mv(A, x), mv(B, x))], "axpby_mv")
    Ah = [[(A[i][j] + u1[i] * v1[j]) + u2[i] * v2[j] for j in range(n)] for i in range(m)]
    gx = [SV_BETA * s_ + z[j] for j, s_ in enumerate(mvt(Ah, yv))]
    gw = [SV_ALPHA * s_ for s_ in mv(Ah, gx)]
    oA, ox, ow = orc.gemver(SV_ALPHA, SV_BETA, ins["A"], ins["u1"], ins["v1"], ins["u2"], ins["v2"], ins["y"],
                            ins["z"])
    _sv_same(oA, [e for row in Ah for e in row], "gemver Ahat")
    _sv_same(ox, gx, "gemver x")
    _sv_same(ow, gw, "gemver w")


def pin_special_values(orc):
    for case in SV_CASES:
        for m, n in SV_SHAPES:
            special_values_case(orc, case, m, n)
    for values in ([1.0, float("inf"), 2.0], [float("inf"), -1.0, -float("inf")], [0.5, float("nan"), 1.0]):
        _sv_same([orc.reduce_sum(np.array(values))], [sum(values)], "reduce_sum")
        other = [float("inf"), -float("inf"), 0.0]
        _sv_same(orc.vector_add(np.array(values), np.array(other)), [p + q for p, q in zip(values, other)],
                 "vector_add")


ALL_PINS = [
    pin_bruteforce_matvec,
    pin_bruteforce_matvec_t,
    pin_bruteforce_ata_x,
    pin_bruteforce_bicg,
    pin_bruteforce_axpby,
    pin_identity_ata,
    pin_adjoint,
    pin_closed_forms,
    pin_integer_exact,
    pin_numpy_crosscheck,
    pin_reduce_sum,
    pin_vector_add,
    pin_gemver,
    pin_special_values,
]
