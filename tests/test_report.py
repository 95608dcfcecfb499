"""Speedup reporting (Sec. 4.1.4) against the averages the paper prints."""
import json
import math
import os

import pytest

from paper_2512_22147_amd import report

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_speedup_tables.json")


def _tables():
    with open(GOLDEN) as f:
        return json.load(f)["tables"]


@pytest.mark.parametrize("name", list(_tables()))
def test_printed_averages_follow_the_fe_only_rule(name):
    t = _tables()[name]
    for col, printed in enumerate(t["average"]):
        vals = [None if r[col] == "Err" else r[col] for r in t["rows"].values()]
        # the printed averages are rounded or truncated to two decimals (5.058 prints as 5.05)
        assert abs(report.average_speedup(vals) - printed) <= 0.01, (name, col)


def test_err_rows_are_excluded_not_zeroed():
    # Table 3, Direct LLM: 1.13 only when dwthaar1d's 'Err' is left out
    t = _tables()["Table 3 (AMD APP SDK, Hygon DCU)"]
    vals = [r[2] for r in t["rows"].values()]
    assert abs(report.average_speedup([None if v == "Err" else v for v in vals]) - 1.13) <= 0.005
    zeroed = sum(0.0 if v == "Err" else v for v in vals) / len(vals)
    assert abs(zeroed - 1.13) > 0.1
    assert math.isnan(report.average_speedup([None, None]))


def test_speedup_and_selection():
    assert report.speedup(2.0, 0.5) == 4.0
    with pytest.raises(ValueError):
        report.speedup(0.0, 1.0)
    res = [(0.20, 0.0, True), (0.10, 1e-7, True), (0.05, 1.0, False)]
    assert report.selection_speedup(res, 1) == pytest.approx(2.0)
    assert report.selection_speedup(res, 2) is None   # failed FE: not counted
    assert report.selection_speedup(res, -1) is None
    assert report.selection_speedup([(float("nan"), 0.0, True)], 0) is None
