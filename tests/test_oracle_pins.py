"""The oracle against what the mathematics and the paper fix (CPU only)."""
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from tests import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(orc, pin):
    pin(orc)


def test_oracle_thread_invariance():
    """Each output is summed by one thread in ascending order, so the result
    is bit-identical for any OpenMP thread count."""
    code = (
        "import numpy as np, oracle\n"
        "from paper_2512_22147_amd import datagen\n"
        "A = datagen.uniform(61, 0, (333, 517), np.float32)\n"
        "x = datagen.uniform(61, 1, (517,), np.float32)\n"
        "y, t = oracle.ata_x(A, x)\n"
        "print(oracle.default().num_threads(), y.tobytes().hex()[:64], hash(y.tobytes()), hash(t.tobytes()))\n"
    )
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    outs = []
    for nt in ("1", "3", "8"):
        env = dict(os.environ, OMP_NUM_THREADS=nt, PYTHONPATH=root, PYTHONHASHSEED="0")
        r = subprocess.run([sys.executable, "-c", code], env=env, cwd=root,
                           capture_output=True, text=True, check=True)
        parts = r.stdout.split()
        assert parts[0] == nt
        outs.append(parts[1:])
    assert outs[0] == outs[1] == outs[2]


# ---- Eq. 3: trimmed mean --------------------------------------------------

def test_trimmed_mean_paper_parameters():
    # R = 30 runs, k = 3 dropped at each end (Sec. 4.1.3): samples 1..30 keep
    # 4..27, whose mean is 15.5.
    assert oracle.trimmed_mean(list(range(1, 31)), 3) == 15.5
    # outliers at both ends are removed
    s = [1.0] * 24 + [0.001, 0.002, 0.003] + [100.0, 200.0, 300.0]
    assert oracle.trimmed_mean(s, 3) == 1.0


def test_trimmed_mean_order_and_ties():
    s = [5.0, 1.0, 3.0]
    assert oracle.trimmed_mean(s, 1) == 3.0
    assert oracle.trimmed_mean(list(reversed(s)), 1) == 3.0
    assert oracle.trimmed_mean([2.0, 2.0, 2.0, 2.0, 7.0], 1) == 2.0
    assert oracle.trimmed_mean([4.0, 8.0], 0) == 6.0


@pytest.mark.parametrize("R,k", [(6, 3), (2, 1), (0, 0), (5, -1)])
def test_trimmed_mean_needs_R_gt_2k(R, k):
    with pytest.raises(ValueError):
        oracle.trimmed_mean([1.0] * R, k)


# ---- Eq. 4: functional equivalence (normwise reading) ----------------------

def test_fe_error_values():
    assert oracle.fe_error([1.0, 2.0, 3.0], [1.0, 2.0, 3.0]) == 0.0
    assert oracle.fe_error([1.0, 2.03, 3.0], [1.0, 2.0, 3.0]) == pytest.approx(0.01)
    assert oracle.fe_error([-3.0], [3.0]) == 2.0
    assert oracle.fe_error([], []) == 0.0
    assert oracle.fe_error([0.0, 0.0], [0.0, 0.0]) == 0.0
    assert oracle.fe_error([0.0, 1e-300], [0.0, 0.0]) == math.inf
    assert oracle.fe_error([1.0, float("nan")], [1.0, 2.0]) == math.inf
    assert oracle.fe_error([1.0, float("inf")], [1.0, 2.0]) == math.inf
    assert oracle.fe_pass([1.0, 2.0001], [1.0, 2.0], 1e-4)
    assert not oracle.fe_pass([1.0, 2.001], [1.0, 2.0], 1e-4)


def test_fe_normwise_not_elementwise():
    # an output near zero may carry a large elementwise error and still be
    # equivalent: the error is measured against the largest reference entry
    assert oracle.fe_error([1000.0, 1e-3 + 1e-5], [1000.0, 1e-3]) < 1e-7


# ---- Eqs. 4-5: next-baseline selection --------------------------------------

def test_select_next():
    assert oracle.select_next([("a", 3.0, True), ("b", 1.0, False), ("c", 2.0, True)]) == "c"
    assert oracle.select_next([("a", 3.0, False)]) is None
    assert oracle.select_next([]) is None
    assert oracle.select_next([("a", 2.0, True), ("b", 2.0, True)]) == "a"


def test_scalar_in_element_type():
    assert oracle.elem_scalar(1.2, np.float32) == float(np.float32(1.2))
    assert oracle.elem_scalar(1.2, np.float64) == 1.2
    assert oracle.elem_scalar(1.5, np.float32) == 1.5
