"""The seeded input generator (Sec. 3.1.2): determinism, ranges, exactness."""
import numpy as np
import pytest

from paper_2512_22147_amd import datagen


def test_splitmix64_known_answer():
    # SplitMix64 seeded with 0 yields these first outputs (Steele, Lea and
    # Flood 2014; the widely published reference sequence).  With the counter
    # form, key(seed, a) is output a of a SplitMix64 seeded with `seed`.
    gamma = 0x9E3779B97F4A7C15
    M = (1 << 64) - 1

    def mix(z):
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M
        return z ^ (z >> 31)

    assert [mix((k * gamma) & M) for k in (1, 2, 3)] == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    # element k of array a: mix(key + (k + 1) gamma), key = mix(seed + (a + 1) gamma)
    key = mix((5 + 2 * gamma) & M)
    want = [mix((key + (k + 1) * gamma) & M) for k in range(4)]
    assert [int(v) for v in datagen.bits(5, 1, 4)] == want


def test_counter_form_is_prefix_and_offset_stable():
    a = datagen.bits(9, 0, 1000)
    b = datagen.bits(9, 0, 10)
    c = datagen.bits(9, 0, 990, first=10)
    assert np.array_equal(a[:10], b)
    assert np.array_equal(a[10:], c)
    assert not np.array_equal(datagen.bits(9, 1, 10), b)
    assert not np.array_equal(datagen.bits(10, 0, 10), b)


@pytest.mark.parametrize("dt,bits", [(np.float32, 23), (np.float64, 52)])
def test_uniform_range_and_grid(dt, bits):
    v = datagen.uniform(3, 0, 200000, dt)
    assert v.dtype == dt
    assert v.min() >= -1.0 and v.max() < 1.0
    # every value is an integer multiple of 2^-bits (exact conversion)
    scaled = v.astype(np.float64) * 2.0**bits
    assert np.array_equal(scaled, np.round(scaled))
    assert abs(float(v.mean())) < 0.01
    assert abs(float(v.var()) - 1.0 / 3.0) < 0.01
    # the same seed gives the same bits
    assert np.array_equal(v, datagen.uniform(3, 0, 200000, dt))


def test_uniform_matches_definition():
    b = datagen.bits(4, 2, 16)
    want32 = ((b >> np.uint64(40)).astype(np.int64) - 2**23).astype(np.float64) * 2.0**-23
    want64 = ((b >> np.uint64(11)).astype(np.int64) - 2**52).astype(np.float64) * 2.0**-52
    assert np.array_equal(datagen.uniform(4, 2, 16, np.float32).astype(np.float64), want32)
    assert np.array_equal(datagen.uniform(4, 2, 16, np.float64), want64)


def test_normal_moments_and_rounding():
    v64 = datagen.normal(2, 0, 400000, np.float64)
    v32 = datagen.normal(2, 0, 400000, np.float32)
    assert abs(float(v64.mean())) < 0.01
    assert abs(float(v64.std()) - 1.0) < 0.01
    assert np.array_equal(v32, v64.astype(np.float32))
    assert np.isfinite(v64).all()


def test_ternary_values():
    t = datagen.ternary(1, 0, 30000, np.float32)
    vals, counts = np.unique(t, return_counts=True)
    assert list(vals) == [-1.0, 0.0, 1.0]
    assert counts.min() > 9000


def test_workloads_sizes():
    w = datagen.WORKLOADS
    assert w["ata_x_16384"].data_bytes(np.float32) == 16384 * 16384 * 4 + 16384 * 4
    assert w["axpby_mv_8192"].alpha == 1.5 and w["axpby_mv_8192"].beta == 1.2
    assert w["matvec_t_1m_x_64"].m == 1048576 and w["matvec_t_1m_x_64"].n == 64
    ins = datagen.make_inputs("ata_x_1024")
    assert ins["A"].shape == (1024, 1024) and ins["x"].shape == (1024,)
    assert np.array_equal(ins["A"].ravel()[:8], datagen.uniform(0, 0, 8, np.float32))


@pytest.mark.parametrize("kind", ["uniform", "normal", "ternary"])
@pytest.mark.parametrize("dt", [np.float32, np.float64])
def test_draws_in_pieces_equal_one_draw(kind, dt):
    """A large array drawn piece by piece (each piece from its first element's
    counter) is bit for bit the array drawn at once."""
    draw = getattr(datagen, kind)
    whole = draw(9, 4, (777, 41), dt)
    cuts = [0, 1, 100, 101, 500, 777]
    parts = [draw(9, 4, (b - a, 41), dt, first=a * 41) for a, b in zip(cuts[:-1], cuts[1:])]
    assert np.array_equal(whole, np.concatenate(parts))
    with pytest.raises(ValueError):
        draw(9, 4, 3, dt, first=-1)
