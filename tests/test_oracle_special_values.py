"""The oracle on NaN and infinities, against brute force (CPU only).

The GPU special-value tests take the oracle's output classes (finite, +inf,
-inf, NaN) as the truth, so the oracle is pinned on its own, case by case
here (and as one pin among those the planted mistakes must fail): every
operation on tiny inputs holding one NaN or infinity (in four cases beside
an exact zero), against the definitions written as plain Python loops over
Python floats, which follow IEEE double arithmetic (0 * inf is NaN, inf -
inf is NaN).  Outputs must agree in class at every position and, where
finite, to within rounding.
"""
import pytest

import oracle
from tests import oracle_pins


def _case_id(case):
    return "+".join(f"{k}-{'zero' if v == 0 else v}" for k, _, v in case)


@pytest.mark.parametrize("shape", oracle_pins.SV_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("case", oracle_pins.SV_CASES, ids=_case_id)
def test_oracle_special_values_against_brute_force(case, shape):
    oracle_pins.special_values_case(oracle.default(), case, *shape)


def test_oracle_sum_and_add_special_values():
    oracle_pins.pin_special_values(oracle.default())
