"""The parity helper's per-element check (CPU only, oracle values).

The normwise FE error measures every output against max|ref|; an output
whose own error scale is far smaller (here: a row or column of A a million
times smaller than the rest) can be wrong by much more than its scale and
still pass it.  The condition-scaled error catches that.  With dense inputs
of one magnitude the condition scales are all far above max|ref|, and the
condition-scaled bound is the looser of the two: it adds a check, it does
not replace the normwise one.  The oracle's exact results rounded to fp32
(a correct GPU result) pass both."""
import numpy as np
import pytest

from tests.gpu_cases import (TOL, assert_parity, condition_scales, cond_bound, diagnostics, make_inputs,
                             oracle_outputs)

# (op, output, the index of A scaled down: "row" i or "col" j)
CASES = [("matvec", "y", "row"), ("axpby_mv", "y", "row"), ("bicg", "q", "row"), ("bicg", "z", "col"),
         ("matvec_t", "z", "col"), ("ata_x", "y", "col")]


@pytest.mark.parametrize("op,out,axis", CASES, ids=[f"{c[0]}-{c[1]}" for c in CASES])
def test_condition_scaled_error_catches_an_output_with_a_small_scale(op, out, axis):
    m, n, dt = 300, 257, np.float32
    ins = make_inputs(op, m, n, dt, seed=31)
    idx = 17
    for name in ("A", "B"):
        if name in ins:
            if axis == "row":
                ins[name][idx, :] *= np.float32(1e-6)
            else:
                ins[name][:, idx] *= np.float32(1e-6)
    ref = oracle_outputs(op, ins, dt)
    scales = condition_scales(op, ins, dt)
    good = {k: v.astype(dt) for k, v in ref.items()}
    assert_parity(op, good, ref, dt, what="rounded", scales=scales, dims=(m, n))
    r = np.asarray(ref[out], np.float64)
    bad = {k: v.copy() for k, v in good.items()}
    bad[out][idx] = np.float32(r[idx] + 1e-6 * np.max(np.abs(r)))
    err, _, cond = diagnostics(bad[out], ref[out], scales[out])
    assert err <= TOL[dt], "the normwise metric does not see this error"
    assert cond > 100 * cond_bound(m, n, dt), (cond, cond_bound(m, n, dt))
    with pytest.raises(AssertionError, match="condition-scaled"):
        assert_parity(op, bad, ref, dt, what="perturbed", scales=scales, dims=(m, n))


def test_condition_scales_are_loose_for_inputs_of_one_magnitude():
    """Dense uniform inputs: every condition scale exceeds max|y| (so the
    normwise check is the tighter one there)."""
    ins = make_inputs("ata_x", 300, 257, np.float32, seed=31)
    y = oracle_outputs("ata_x", ins, np.float32)["y"]
    sc = condition_scales("ata_x", ins, np.float32)["y"]
    assert float(np.min(sc)) > float(np.max(np.abs(y)))
