"""The C-ABI library on the host: symbols, argument checks, host logic.

No kernel runs here: every call below either is host-only (Eq. 3, the FE
metric, workspace sizing) or fails its argument checks before anything is
launched.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2512_22147_amd import mep

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mep.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mep_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return mep.lib()


def test_library_exports_every_declared_function(L):
    names = declared_functions()
    assert len(names) == 24
    for name in names:
        assert hasattr(L, name), f"{name} not exported"
    assert sorted(mep.EXPORTS) == names


def test_version(L):
    assert "gfx950" in mep.mep_version()


def test_trimmed_mean_matches_eq3():
    rng = np.random.default_rng(5)
    for R, k in [(30, 3), (7, 0), (5, 2), (31, 15)]:
        s = list(rng.exponential(1.0, R))
        assert mep.mep_trimmed_mean(s, k) == oracle.trimmed_mean(s, k)
    assert mep.mep_trimmed_mean(list(range(1, 31)), 3) == 15.5
    assert math.isnan(mep.mep_trimmed_mean([1.0] * 6, 3))
    assert math.isnan(mep.mep_trimmed_mean([1.0] * 6, -1))


@pytest.mark.parametrize("dt", [np.float32, np.float64])
def test_check_fe_matches_metric(dt):
    rng = np.random.default_rng(7)
    ref = rng.standard_normal(1000)
    for scale in (0.0, 1e-9, 1e-5, 1e-2):
        out = (ref + scale * rng.standard_normal(1000)).astype(dt)
        err, ok = mep.mep_check_fe(out, ref, 1e-4)
        want = oracle.fe_error(out, ref)
        assert err == pytest.approx(want, rel=1e-12, abs=0.0)
        assert ok == (want <= 1e-4)
    bad = ref.astype(dt).copy()
    bad[17] = np.nan
    assert mep.mep_check_fe(bad, ref, 1.0) == (math.inf, False)
    assert mep.mep_check_fe(np.zeros(4, dt), np.zeros(4), 0.0) == (0.0, True)
    assert mep.mep_check_fe(np.array([0, 1e-30], dt), np.zeros(2), 1.0)[1] is False
    assert mep.mep_check_fe(np.zeros(0, dt), np.zeros(0), 0.0) == (0.0, True)
    # a non-finite reference is refused: max() would skip a NaN entry, and an
    # all-NaN reference would otherwise pass every output
    for v in (np.nan, np.inf):
        badref = ref.copy()
        badref[3] = v
        with pytest.raises(mep.MepError, match="not finite"):
            mep.mep_check_fe(ref.astype(dt), badref, 1.0)
    with pytest.raises(mep.MepError):
        mep.mep_check_fe(np.zeros(4, dt), np.full(4, np.nan), 1.0)


def test_workspace_sizes():
    f32, f64 = mep.MEP_F32, mep.MEP_F64
    ws = mep.mep_workspace_bytes
    assert ws(mep.MEP_OP_MATVEC, f32, 1000, 1000) == 0           # one panel: no partials
    assert ws(mep.MEP_OP_ATA_X, f32, 16384, 16384) >= 256 * 16384 * 4
    assert ws(mep.MEP_OP_ATA_X, f32, 0, 100) == 0
    assert ws(mep.MEP_OP_ATA_X, f32, 100, 0) == 0
    assert ws(mep.MEP_OP_MATVEC_T, f64, 1 << 20, 64) > 0
    assert ws(mep.MEP_OP_ATA_X, f64, 1000, 40000) > 1000 * 8    # two passes keep t
    assert ws(99, f32, 10, 10) == 0
    assert ws(mep.MEP_OP_MATVEC, 7, 10, 10) == 0
    for op in range(5):
        for dt in (f32, f64):
            assert mep.mep_variant_count(op, dt, 4096, 4096) >= 1
    assert mep.mep_variant_count(9, f32, 10, 10) == 0
    assert mep.mep_workspace_bytes(mep.MEP_OP_REDUCE_SUM, f32, 1, 1 << 28) >= 512 * 4
    assert mep.mep_workspace_bytes(mep.MEP_OP_REDUCE_SUM, f32, 1, 0) == 0
    assert mep.mep_workspace_bytes(mep.MEP_OP_VECTOR_ADD, f64, 1, 1000) == 0
    assert mep.mep_variant_count(mep.MEP_OP_REDUCE_SUM, f32, 1, 1000) == 1
    assert mep.mep_variant_count(mep.MEP_OP_VECTOR_ADD, f32, 1, 1000) == 6
    assert "chunks" in mep.mep_variant_info(mep.MEP_OP_VECTOR_ADD, f32, 1, 1000, 2)
    assert "buffer rows" in mep.mep_variant_info(mep.MEP_OP_VECTOR_ADD, f32, 1, 1000, 0)
    with pytest.raises(mep.MepError):
        mep.mep_variant_info(mep.MEP_OP_VECTOR_ADD, f32, 1, 1000, 6)
    # GEMVER: pass 1 column partials or pass 2 dot partials, whichever is larger
    assert ws(mep.MEP_OP_GEMVER, f32, 16384, 16384) >= 64 * 16384 * 4
    assert ws(mep.MEP_OP_GEMVER, f64, 0, 100) == 0
    assert ws(mep.MEP_OP_GEMVER, f64, 100, 0) == 0
    for dt in (f32, f64):
        for m, n in [(1, 1), (7, 1), (1, 7), (3, 5), (129, 16384), (67, 40000), (4096, 4096)]:
            assert mep.mep_variant_count(mep.MEP_OP_GEMVER, dt, m, n) >= 1
            assert ws(mep.MEP_OP_GEMVER, dt, m, n) >= ws(mep.MEP_OP_MATVEC, dt, m, n)
    info = mep.mep_variant_info(mep.MEP_OP_ATA_X, f32, 16384, 16384, 0)
    assert "G=512" in info and "nt" in info
    with pytest.raises(mep.MepError):
        mep.mep_variant_info(mep.MEP_OP_ATA_X, f32, 16384, 16384, 99)


# Default shapes measured on MI355X (candidate sweeps over row lengths, element
# types, operations, streamed 1 GiB and cache-resident 32-64 MiB matrices):
# (op, dtype, m, n) -> the shape candidate 0 must have.  A change of the rule
# has to come with a sweep that justifies it.
MEASURED_DEFAULTS = [
    # the benchmark workloads
    ("ATA_X", 0, 16384, 16384, "G=512 V=8 B=2 WPE=2 nt rotated cus=24/32"),
    ("ATA_X", 1, 16384, 16384, "G=512 V=16 B=1 WPE=2 nt rotated cus=26/32"),
    ("ATA_X", 0, 1024, 1024, "G=64 V=4 B=2 WPE=4 nt"),
    ("BICG", 0, 4096, 4096, "G=512 V=2 B=8 WPE=2 nt cyclic cus=32/32"),
    ("AXPBY_MV", 0, 8192, 8192, "G=512 V=8 B=1 WPE=2 nt cyclic cus=32/32"),
    ("MATVEC_T", 0, 1 << 20, 64, "G=16 V=1 B=8 WPE=4 nt cyclic cus=16/32"),
    ("GEMVER", 0, 16384, 16384, "G=1024 V=4 B=2 WPE=4 nt cyclic cus=32/32"),
    ("MATVEC", 0, 16384, 16384, "G=512 V=8 B=2 WPE=2 nt rotated cus=24/32"),
    # other row lengths, streamed
    ("ATA_X", 0, 65536, 4096, "G=512 V=2 B=8 WPE=2 nt cyclic cus=24/32"),
    ("MATVEC_T", 0, 131072, 2048, "G=512 V=2 B=8 WPE=2 nt"),
    ("MATVEC", 0, 131072, 2048, "G=512 V=2 B=4 WPE=4 nt"),
    ("BICG", 1, 131072, 1024, "G=512 V=1 B=8 WPE=4 nt"),
    ("MATVEC", 0, 32768, 8192, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("BICG", 0, 32768, 8192, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("MATVEC_T", 0, 32768, 8192, "G=512 V=8 B=2 WPE=2 nt cyclic cus=32/32"),
    ("AXPBY_MV", 0, 8192, 16384, "G=512 V=8 B=1 WPE=2 nt cyclic cus=24/32"),
    ("GEMVER", 0, 131072, 2048, "G=512 V=2 B=8 WPE=2 nt"),
    ("GEMVER", 1, 131072, 1024, "G=256 V=4 B=2 WPE=4 nt"),
    # streamed fp32 rows past 2816 vectors, and fp64 ATAX rows past 5632
    # vectors: the rotated block map; the rest keep the cyclic one
    ("MATVEC_T", 0, 20000, 15000, "G=512 V=8 B=2 WPE=2 nt rotated cus=24/32"),
    ("BICG", 0, 22000, 12200, "G=512 V=8 B=2 WPE=2 nt rotated cus=24/32"),
    ("MATVEC", 0, 27000, 10000, "G=512 V=8 B=2 WPE=2 nt cyclic cus=24/32"),
    ("ATA_X", 1, 16000, 8000, "G=512 V=8 B=2 WPE=2 nt cyclic cus=22/32"),
    ("ATA_X", 1, 14000, 14000, "G=512 V=16 B=1 WPE=2 nt rotated cus=26/32"),
    ("BICG", 1, 16384, 16384, "G=512 V=16 B=1 WPE=2 nt cyclic cus=26/32"),
    # narrow rows: as many lanes per row as the row has vectors
    ("MATVEC", 0, 1 << 24, 12, "G=4 V=1 B=8 WPE=4 nt cyclic cus=32/32"),
    ("ATA_X", 1, 1 << 24, 8, "G=4 V=1 B=8 WPE=4 nt"),
    ("MATVEC_T", 0, 1 << 24, 32, "G=8 V=1 B=8 WPE=4 nt"),
    ("BICG", 0, 1 << 25, 8, "G=2 V=1 B=4 WPE=4 nt"),
    ("BICG", 1, 1 << 24, 8, "G=4 V=1 B=4 WPE=4 nt"),
    ("BICG", 0, 1 << 20, 4, "G=2 V=1 B=8 WPE=4 cached"),
    ("MATVEC_T", 1, 1 << 24, 8, "G=4 V=1 B=8 WPE=4 nt"),
    ("BICG", 1, 1 << 22, 32, "G=16 V=1 B=4 WPE=4 nt"),
    # rows between the measured lengths: the smallest 512-lane shape that covers them
    ("ATA_X", 0, 65472, 4100, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("BICG", 0, 87267, 3076, "G=512 V=2 B=8 WPE=2 nt"),
    ("ATA_X", 0, 21838, 12292, "G=512 V=8 B=2 WPE=2 nt rotated cus=24/32"),
    ("MATVEC_T", 0, 13107, 20480, "G=512 V=16 B=1 WPE=2 nt cyclic cus=26/32"),
    ("BICG", 0, 13107, 20480, "G=512 V=16 B=1 WPE=2 nt cyclic cus=32/32"),
    ("ATA_X", 1, 10922, 12288, "G=512 V=16 B=1 WPE=2 nt rotated cus=26/32"),
    ("MATVEC", 0, 1024, 20480, "G=1024 V=8 B=1 WPE=4 nt"),
    # cache-resident
    ("MATVEC", 0, 4096, 2048, "G=256 V=2 B=4 WPE=4 nt"),
    ("ATA_X", 0, 4096, 2048, "G=512 V=2 B=8 WPE=2 nt"),
    ("AXPBY_MV", 0, 2048, 4096, "G=256 V=4 B=1 WPE=4 nt"),
    ("MATVEC", 0, 1024, 16384, "G=512 V=8 B=2 WPE=2 nt cyclic cus=32/32"),
    ("BICG", 0, 1024, 16384, "G=512 V=8 B=2 WPE=2 cached"),
    ("MATVEC", 0, 6553, 2560, "G=256 V=4 B=2 WPE=4 nt"),
    ("MATVEC_T", 0, 5461, 3072, "G=512 V=2 B=8 WPE=2 nt"),
    ("MATVEC_T", 0, 4096, 6144, "G=512 V=4 B=4 WPE=2 cached"),
    ("ATA_X", 0, 2340, 7168, "G=512 V=4 B=4 WPE=2 cached"),
    ("BICG", 0, 13107, 1280, "G=512 V=1 B=8 WPE=4 nt"),
    ("MATVEC", 1, 2340, 3584, "G=512 V=4 B=4 WPE=2 nt"),
    # 257-512-vector rows on 512-vector shapes
    ("MATVEC", 0, 209715, 1280, "G=512 V=1 B=8 WPE=4 nt"),
    ("ATA_X", 1, 209715, 640, "G=512 V=1 B=8 WPE=4 nt"),
    ("AXPBY_MV", 0, 104857, 1280, "G=512 V=1 B=4 WPE=4 nt"),
    # streamed rows that fill their group: the next wider shape
    ("MATVEC", 0, 74898, 3584, "G=512 V=4 B=4 WPE=2 nt cyclic cus=32/32"),
    ("MATVEC", 0, 65536, 4096, "G=512 V=2 B=8 WPE=2 nt cyclic cus=24/32"),
    ("BICG", 0, 74898, 3584, "G=512 V=2 B=8 WPE=2 nt"),
    ("ATA_X", 1, 37449, 3584, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("BICG", 0, 37449, 7168, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("BICG", 0, 52428, 5120, "G=512 V=4 B=4 WPE=2 nt cyclic cus=32/32"),
    ("MATVEC_T", 0, 37449, 7168, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("MATVEC", 0, 43690, 6144, "G=512 V=4 B=4 WPE=2 nt cyclic cus=24/32"),
    ("MATVEC_T", 0, 1 << 23, 320, "G=64 V=2 B=4 WPE=4 nt"),
    ("ATA_X", 0, 1 << 21, 512, "G=64 V=4 B=2 WPE=4 nt"),
]


@pytest.mark.parametrize("op,dt,m,n,want", MEASURED_DEFAULTS,
                         ids=[f"{c[0]}-{'f32' if c[1] == 0 else 'f64'}-{c[2]}x{c[3]}" for c in MEASURED_DEFAULTS])
def test_measured_default_shapes(op, dt, m, n, want):
    info = mep.mep_variant_info(getattr(mep, f"MEP_OP_{op}"), dt, m, n, 0)
    assert want in info, info


def _rc(fn, *args):
    rc = fn(*args)
    return rc, mep.mep_last_error()


FAKE = 1 << 20  # an aligned address that is never dereferenced: the checks fail first


def test_argument_errors(L):
    f32 = mep.MEP_F32
    rc, msg = _rc(L.mep_matvec, 3, 4, 4, FAKE, FAKE, FAKE * 2, None, 0, None)
    assert rc == mep.MEP_EINVAL and "dtype" in msg
    rc, msg = _rc(L.mep_matvec, f32, -1, 4, FAKE, FAKE, FAKE * 2, None, 0, None)
    assert rc == mep.MEP_EINVAL and "negative" in msg
    rc, msg = _rc(L.mep_matvec, f32, 1 << 31, 4, FAKE, FAKE, FAKE * 2, None, 0, None)
    assert rc == mep.MEP_EINVAL
    rc, msg = _rc(L.mep_matvec, f32, 4, 4, None, FAKE, FAKE * 2, None, 0, None)
    assert rc == mep.MEP_EINVAL and "A" in msg
    rc, msg = _rc(L.mep_matvec, f32, 4, 4, FAKE + 2, FAKE * 4, FAKE * 2, None, 0, None)
    assert rc == mep.MEP_EALIGN
    rc, msg = _rc(L.mep_matvec, mep.MEP_F64, 4, 4, FAKE + 4, FAKE * 4, FAKE * 2, None, 0, None)
    assert rc == mep.MEP_EALIGN
    # output overlapping an input
    rc, msg = _rc(L.mep_matvec, f32, 4, 4, FAKE, FAKE * 4, FAKE + 8, None, 0, None)
    assert rc == mep.MEP_EINVAL and "overlap" in msg
    # workspace too small
    need = mep.mep_workspace_bytes(mep.MEP_OP_ATA_X, f32, 4096, 4096)
    rc, msg = _rc(L.mep_ata_x, f32, 4096, 4096, FAKE, FAKE * 64, FAKE * 65, None, FAKE * 128,
                  need - 1, None)
    assert rc == mep.MEP_EWORKSPACE
    rc, msg = _rc(L.mep_ata_x, f32, 4096, 4096, FAKE, FAKE * 64, FAKE * 65, None, None, need, None)
    assert rc == mep.MEP_EWORKSPACE
    rc, msg = _rc(L.mep_ata_x, f32, 4096, 4096, FAKE, FAKE * 64, FAKE * 65, None, FAKE * 128 + 16,
                  need, None)
    assert rc == mep.MEP_EALIGN
    # BICG needs p and q together
    rc, msg = _rc(L.mep_matvec_t, f32, 8, 8, FAKE, FAKE * 4, FAKE * 5, FAKE * 6, None, None, 0, None)
    assert rc == mep.MEP_EINVAL and "p and q" in msg
    rc, msg = _rc(L.mep_matvec_t, f32, 8, 8, FAKE, FAKE * 4, FAKE * 5, None, FAKE * 6, None, 0, None)
    assert rc == mep.MEP_EINVAL and "p and q" in msg
    # two outputs overlapping each other
    wsb = mep.mep_workspace_bytes(mep.MEP_OP_BICG, f32, 8, 8)
    rc, msg = _rc(L.mep_matvec_t, f32, 8, 8, FAKE, FAKE * 4, FAKE * 5, FAKE * 6, FAKE * 5 + 16,
                  FAKE * 128, wsb, None)
    assert rc == mep.MEP_EINVAL and "overlap" in msg
    rc, msg = _rc(L.mep_axpby_mv, f32, 8, 8, 1.0, FAKE, 1.0, None, FAKE * 4, FAKE * 5, None, 0, None)
    assert rc == mep.MEP_EINVAL and "B" in msg
    rc, msg = _rc(L.mep_reduce_sum, f32, 1000, FAKE, FAKE * 4, None, 0, None)
    assert rc == mep.MEP_EWORKSPACE
    rc, msg = _rc(L.mep_reduce_sum, f32, 1000, None, FAKE * 4, FAKE * 8, 1 << 16, None)
    assert rc == mep.MEP_EINVAL
    rc, msg = _rc(L.mep_vector_add, f32, 1000, FAKE, FAKE * 2, FAKE + 64, None)
    assert rc == mep.MEP_EINVAL and "overlap" in msg
    rc, msg = _rc(L.mep_vector_add, mep.MEP_F64, 10, FAKE, FAKE * 2, FAKE * 3 + 4, None)
    assert rc == mep.MEP_EALIGN
    # GEMVER: Ahat may be A itself but must not overlap it otherwise
    gw = mep.mep_workspace_bytes(mep.MEP_OP_GEMVER, f32, 64, 64)
    vecs = [FAKE * k for k in range(4, 12)]  # u1, v1, u2, v2, y, z, x, w
    rc, msg = _rc(L.mep_gemver, f32, 64, 64, 1.0, 1.0, FAKE, FAKE + 64, *vecs, FAKE * 16, gw, None)
    assert rc == mep.MEP_EINVAL and "overlap" in msg
    rc, msg = _rc(L.mep_gemver, f32, 64, 64, 1.0, 1.0, FAKE, FAKE * 2, *vecs[:6], None, vecs[7],
                  FAKE * 16, gw, None)
    assert rc == mep.MEP_EINVAL and "x" in msg
    rc, msg = _rc(L.mep_gemver, f32, 64, 64, 1.0, 1.0, FAKE, FAKE * 2, *vecs, FAKE * 16, gw - 1, None)
    assert rc == mep.MEP_EWORKSPACE
    rc, msg = _rc(L.mep_gemver, mep.MEP_F64, 64, 64, 1.0, 1.0, FAKE, FAKE * 2, FAKE * 4 + 4, *vecs[1:],
                  FAKE * 16, gw, None)
    assert rc == mep.MEP_EALIGN
    # an output on an input vector
    rc, msg = _rc(L.mep_gemver, f32, 64, 64, 1.0, 1.0, FAKE, FAKE * 2, *vecs[:6], vecs[5], vecs[7],
                  FAKE * 16, gw, None)
    assert rc == mep.MEP_EINVAL and "overlap" in msg


MAX_M = 1 << 30
MAX_N = 65535 * 8192


@pytest.mark.parametrize("which", ["m", "n"])
def test_size_limits_are_exact(L, which):
    """The largest accepted sizes (m = 2^30 rows, rows of 65535 * 8192
    elements) pass the size check and one more fails it.  A is given one
    byte off its element alignment, so an accepted size stops at the next
    check (MEP_EALIGN) and nothing is ever launched."""
    bad_a = FAKE + 1
    for dt in (mep.MEP_F32, mep.MEP_F64):
        for size, want in ((MAX_M if which == "m" else MAX_N, mep.MEP_EALIGN),
                           ((MAX_M if which == "m" else MAX_N) + 1, mep.MEP_EINVAL)):
            m, n = (size, 1) if which == "m" else (1, size)
            rc, msg = _rc(L.mep_matvec, dt, m, n, bad_a, FAKE, FAKE, None, 0, None)
            assert rc == want, (dt, m, n, msg)
            rc, msg = _rc(L.mep_ata_x, dt, m, n, bad_a, FAKE, FAKE, None, None, 0, None)
            assert rc == want, (dt, m, n, msg)
            rc, msg = _rc(L.mep_ata_x_noalloc, dt, m, n, bad_a, FAKE, FAKE, None, None)
            assert rc == want, (dt, m, n, msg)
            if want == mep.MEP_EINVAL:
                assert "2^30" in msg or "row length" in msg, msg


def test_harness_errors(L):
    c = mep.MepCall()
    c.op, c.dtype, c.m, c.n = mep.MEP_OP_ATA_X, mep.MEP_F32, 8, 8
    mean = ctypes.c_double()
    for R, k in [(6, 3), (2, 1), (0, 0)]:
        assert L.mep_time_trimmed(ctypes.byref(c), 0, R, k, 1, 0, ctypes.byref(mean), None) == mep.MEP_EBUDGET
    assert L.mep_time_trimmed(ctypes.byref(c), 0, 30, 3, 0, 0, ctypes.byref(mean), None) == mep.MEP_EBUDGET
    assert L.mep_time_trimmed(None, 0, 30, 3, 1, 0, ctypes.byref(mean), None) == mep.MEP_EINVAL
    c.op = 42
    assert L.mep_run(ctypes.byref(c)) == mep.MEP_EINVAL
    c.op = mep.MEP_OP_BICG
    assert L.mep_run(ctypes.byref(c)) == mep.MEP_EINVAL
    assert L.mep_set_variant(17, 0) == mep.MEP_EINVAL
    assert L.mep_profile_begin(0) == mep.MEP_EINVAL
    assert L.mep_profile_begin_sampled(4, 0, 1) == mep.MEP_EINVAL
    assert L.mep_profile_begin_sampled(4, 1, 0) == mep.MEP_EINVAL
    assert L.mep_profile_begin_sampled(0, 1, 1) == mep.MEP_EINVAL
    assert L.mep_profile_end(None, None) == mep.MEP_EINVAL
    assert L.mep_stream_copy(FAKE, FAKE * 2, 24, None) == mep.MEP_EALIGN
    assert L.mep_stream_copy(FAKE, FAKE + 16, 64, None) == mep.MEP_EINVAL
    assert L.mep_stream_copy(None, None, 0, None) == mep.MEP_OK
    best = ctypes.c_int()
    c.op = mep.MEP_OP_ATA_X
    assert L.mep_select_variant(ctypes.byref(c), 0, 4, 2, 1, 0, 1e-4, 0, ctypes.byref(best), None, 0) == mep.MEP_EBUDGET
    assert L.mep_select_variant(None, 0, 30, 3, 1, 0, 1e-4, 0, ctypes.byref(best), None, 0) == mep.MEP_EINVAL
    c.op, c.A, c.out2 = mep.MEP_OP_GEMVER, FAKE, FAKE
    assert L.mep_select_variant(ctypes.byref(c), 0, 30, 3, 1, 0, 1e-4, 0, ctypes.byref(best), None, 0) == mep.MEP_EINVAL
    assert "out-of-place" in mep.mep_last_error()
    c.A = c.out2 = None
    # a flush buffer that is not a whole number of 16-byte vectors, or not
    # 16-byte aligned, is refused before anything runs
    c.op = mep.MEP_OP_ATA_X
    c.flush_buf, c.flush_bytes = FAKE, 1000
    assert L.mep_select_variant(ctypes.byref(c), 0, 30, 3, 1, 0, 1e-4, 0, ctypes.byref(best), None, 0) == mep.MEP_EALIGN
    c.flush_buf, c.flush_bytes = FAKE + 8, 1024
    assert L.mep_select_variant(ctypes.byref(c), 0, 30, 3, 1, 0, 1e-4, 0, ctypes.byref(best), None, 0) == mep.MEP_EALIGN
    c.flush_buf, c.flush_bytes = None, 0
    c.op = 77
    assert L.mep_select_variant(ctypes.byref(c), 0, 30, 3, 1, 0, 1e-4, 0, ctypes.byref(best), None, 0) == mep.MEP_EINVAL


def test_noalloc_refuses_beyond_its_scratch_before_any_launch(L):
    """mep_ata_x_noalloc checks its plan's scratch need before touching a
    device: 2^23 rows of 40000 fp32 (two-pass path) need more than 64 MiB.
    The pointers are never dereferenced."""
    import ctypes

    base = 1 << 40
    rc = L.mep_ata_x_noalloc(mep.MEP_F32, 1 << 23, 40000, ctypes.c_void_p(base),
                             ctypes.c_void_p(base + (1 << 42)), ctypes.c_void_p(base + (1 << 43)), None, None)
    assert rc == mep.MEP_EWORKSPACE
    assert str(mep.NOALLOC_SCRATCH_BYTES) in mep.mep_last_error()
    assert L.mep_ata_x_noalloc(mep.MEP_F32, 4, 4, None, None, None, None, None) == mep.MEP_EINVAL
    assert L.mep_ata_x_noalloc(9, 4, 4, None, None, None, None, None) == mep.MEP_EINVAL
