"""The sum's parity bound can fail (CPU only, against the oracle's values).

On the benchmark's sum inputs (2^28 non-negative fp32 terms) an all-zero
result, and a result missing any one workgroup's partial, both lie outside the
bound the GPU test applies (min(1e-4, gamma_d) relative error, d from the
kernel's summation depth): the GPU test cannot pass a sum that drops work.
"""
import numpy as np

import oracle
from paper_2512_22147_amd import datagen
from tests.sum_bound import sum_chunks, sum_depth, sum_error_bound


def test_depth_of_the_benchmark_sum():
    # 2^26 vectors over 512 workgroups: chunks of 2^17 vectors, 512 per lane
    assert sum_chunks(1 << 28, np.float32) == (512, 1 << 17, 4)
    assert sum_depth(1 << 28, np.float32) == 512 + 64
    assert 3.4e-5 < sum_error_bound(1 << 28, np.float32) < 3.5e-5
    # fp64: the oracle's own sequential error dominates (gamma_(n-1) in fp64)
    assert sum_error_bound(1 << 20, np.float64) > (1 << 20) * 2.0**-53
    # the element-wise path (x off a 16-byte boundary) has 4x longer lane chains
    assert sum_depth(1 << 28, np.float32, offset=1) == 2048 + 64
    assert sum_chunks(0, np.float64) == (1, 0, 2)


def test_zero_and_dropped_partial_fail_on_the_benchmark_inputs():
    x = datagen.make_inputs("reduce_sum_256m")["x"]
    assert x.dtype == np.float32 and float(x.min()) >= 0.0
    bound = min(1e-4, sum_error_bound(x.size, np.float32))
    # the oracle's sum of each workgroup's chunk (the chunks cover x once);
    # the total is their sum, within 1e-13 of the oracle's whole-vector value
    # (one fp64 sum of 512 non-negative terms), far inside the bound
    nb, chunk, vw = sum_chunks(x.size, np.float32)
    assert nb * chunk * vw == x.size
    parts = [oracle.reduce_sum(x[b * chunk * vw:(b + 1) * chunk * vw]) for b in range(nb)]
    ref = sum(parts)
    # an all-zero output
    assert abs(0.0 - ref) / abs(ref) > bound
    # every result that misses one workgroup's chunk
    smallest = min(parts)
    assert smallest / abs(ref) > 10 * bound, (smallest / abs(ref), bound)
