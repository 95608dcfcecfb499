"""Planted mistakes in copies of the oracle must each fail at least one pin.

Each mutant is a textual edit of ``oracle/oracle.c`` (a dropped term, a wrong
sign or index, a transposed operand, a lower-precision accumulator, a swapped
operand), compiled with gcc into a temporary directory and checked in a
subprocess, so a mutant that reads out of bounds cannot take pytest down.
The real oracle is never modified.
"""
import json
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "matvec_drops_last_term": (
        "for (int64_t j = 0; j < n; ++j)\n            acc += A[i * n + j] * x[j];",
        "for (int64_t j = 0; j < n - 1; ++j)\n            acc += A[i * n + j] * x[j];"),
    "matvec_column_major_read": (
        "acc += A[i * n + j] * x[j];", "acc += A[j * m + i] * x[j];"),
    "matvec_fp32_accumulator": ("double acc = 0.0;", "float acc = 0.0f;"),
    "matvec_t_wrong_sign": ("z[j] += A[i * n + j] * w[i];", "z[j] -= A[i * n + j] * w[i];"),
    "matvec_t_off_by_one_weight": ("z[j] += A[i * n + j] * w[i];",
                                   "z[j] += A[i * n + j] * w[(i + 1) % m];"),
    "ata_x_reuses_x": ("oracle_matvec_t(m, n, A, tt, y);", "oracle_matvec_t(m, n, A, x, y);"),
    "ata_x_rounds_t_to_fp32": (
        "oracle_matvec(m, n, A, x, tt);",
        "oracle_matvec(m, n, A, x, tt);\n    for (int64_t i = 0; i < m; ++i) tt[i] = (double)(float)tt[i];"),
    "bicg_uses_p_for_s": ("oracle_matvec_t(m, n, A, r, s);", "oracle_matvec_t(m, n, A, p, s);"),
    "axpby_same_dot_twice": ("y[i] = alpha * da + beta * db;", "y[i] = alpha * da + beta * da;"),
    "axpby_swapped_scalars": ("y[i] = alpha * da + beta * db;", "y[i] = alpha * db + beta * da;"),
    "axpby_reads_A_for_B": ("db += B[i * n + j] * x[j];", "db += A[i * n + j] * x[j];"),
    "reduce_skips_first": ("for (int64_t i = 0; i < n; ++i)\n        s += x[i];",
                           "for (int64_t i = 1; i < n; ++i)\n        s += x[i];"),
    "reduce_fp32_accumulator": ("double s = 0.0;", "float s = 0.0f;"),
    "vector_add_subtracts": ("c[i] = a[i] + b[i];", "c[i] = a[i] - b[i];"),
    "gemver_drops_second_update": ("Ahat[i * n + j] = (A[i * n + j] + u1[i] * v1[j]) + u2[i] * v2[j];",
                                   "Ahat[i * n + j] = A[i * n + j] + u1[i] * v1[j];"),
    "gemver_w_from_A": ("oracle_matvec(m, n, Ahat, x, w);", "oracle_matvec(m, n, A, x, w);"),
    "gemver_x_misses_z": ("x[j] = beta * x[j] + z[j];", "x[j] = beta * x[j];"),
    "gemver_swapped_scalars": ("w[i] = alpha * w[i];", "w[i] = beta * w[i];"),
    # zero terms skipped: the same result on finite inputs, but 0 * inf must give NaN
    "matvec_skips_zero_elements": ("            acc += A[i * n + j] * x[j];",
                                   "            if (A[i * n + j] != 0.0) acc += A[i * n + j] * x[j];"),
    "matvec_t_skips_zero_weights": ("                z[j] += A[i * n + j] * w[i];",
                                    "                if (w[i] != 0.0) z[j] += A[i * n + j] * w[i];"),
}

RUNNER = r"""
import json, sys, traceback
sys.path.insert(0, sys.argv[2])
import oracle
from tests import oracle_pins
orc = oracle.Oracle(sys.argv[1])
res = {}
for pin in oracle_pins.ALL_PINS:
    try:
        pin(orc)
        res[pin.__name__] = "pass"
    except AssertionError as e:
        res[pin.__name__] = "FAIL: " + str(e)[:200]
    except Exception as e:
        res[pin.__name__] = "ERROR: " + repr(e)[:200]
print(json.dumps(res))
"""


@pytest.fixture(scope="module")
def source():
    with open(oracle.SOURCE) as f:
        return f.read()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, source, tmp_path):
    old, new = MUTANTS[name]
    assert source.count(old) == 1, f"mutation anchor for {name} not unique"
    src = tmp_path / "oracle_mutant.c"
    src.write_text(source.replace(old, new))
    lib = oracle.build(str(src), str(tmp_path / "liboracle_mutant.so"))
    env = dict(os.environ, OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-c", RUNNER, lib, ROOT], env=env, cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        # a crash of the mutant (e.g. an out-of-bounds read) is also a catch
        return
    res = json.loads(r.stdout.strip().splitlines()[-1])
    failed = [k for k, v in res.items() if v != "pass"]
    assert failed, f"mutant {name} passed every pin"
