"""bench.py's output contract on the GPU: one JSON line whose figures agree
with each other (value from the step time and the algorithmic bytes,
roofline fraction from the kernel time, the oracle's CPU baseline present,
the headline output within the fp32 tolerance of the oracle)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line_is_consistent():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    steps, warmup = 16, 2
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--steps", str(steps),
                        "--warmup", str(warmup), "--no-f64", "--no-eq3", "--no-ceiling"],
                       capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    assert d["n_gpus"] == 1 and d["steps"] == steps and d["warmup"] == warmup
    assert d["unit"] == "GB/s" and d["higher_is_better"] is True and d["dtype"] == "f32"
    assert d["data"] == "synthetic" and d["vs_baseline"] is None
    m, n, es = d["config"]["m"], d["config"]["n"], 4
    assert (m, n) == (16384, 16384)
    # value = algorithmic bytes of the whole step (A once, x read, y written) / step time
    step_bytes = (m * n + 2 * n) * es
    assert d["value"] == pytest.approx(step_bytes / (d["ms_per_step"] * 1e-3) / 1e9, rel=2e-3)
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["peak"] == 8000.0 and roof["unit"] == "GB/s"
    assert roof["alg_bytes_per_launch"] == (m * n + n) * es
    assert roof["achieved"] == pytest.approx(roof["alg_bytes_per_launch"] / (roof["kernel_ms"] * 1e-3) / 1e9,
                                             rel=2e-3)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], abs=2e-4)
    # the kernel is at most the step; neither exceeds the HBM peak
    assert roof["kernel_ms"] <= d["ms_per_step"] * 1.02
    assert 0 < d["value"] < 8000.0 and 0 < roof["achieved"] < 8000.0
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == "GB/s" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert d["fe_error_vs_oracle"] <= 1e-4
    fe = d["fe_vs_oracle"]
    assert fe["normwise"] == d["fe_error_vs_oracle"] and fe["pass"] is True
    # the diagnostics beside it: the condition-scaled error is within the
    # rigorous bound 2 gamma_(m+n+64) of any summation order (~3.9e-3 here)
    assert 0 <= fe["condition_scaled"] < 2 * (m + n + 64) * 2.0**-24
    assert fe["elementwise"] >= 0
    assert len(d["other_configs"]) == 4
    for o in d["other_configs"]:
        assert o["ms_per_step"] > 0 and o["kernel_gbs"] > 0 and o["same_size_read_gbs"] > 0
        assert o["kernel_frac_of_read"] == pytest.approx(o["kernel_gbs"] / o["same_size_read_gbs"], rel=2e-3)
