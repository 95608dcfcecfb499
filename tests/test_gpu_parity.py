"""GPU kernels (through the C-ABI) against the CPU oracle.

Bar: normwise relative error <= 1e-4 (fp32) / 1e-12 (fp64) on random inputs;
bit-exact on integer-valued inputs, where every partial sum is an exact
integer in either precision; bitwise run-to-run reproducibility.
"""
import numpy as np
import pytest

from tests.gpu_cases import (OPS, assert_parity, condition_scales, gpu_outputs, make_inputs, op_code,
                             oracle_outputs)

pytestmark = pytest.mark.gpu

DTYPES = [np.float32, np.float64]


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_22147_amd import mep

    for op in range(8):
        mep.mep_set_variant(op, -1)
    yield
    for op in range(8):
        mep.mep_set_variant(op, -1)


# shapes chosen to cover every row-group width, ragged tails of rows and of
# row vectors, several workgroups and several tiles
EDGE_SHAPES = [(1, 1), (1, 7), (7, 1), (3, 5), (63, 63), (64, 64), (65, 129), (100, 1000),
               (257, 4100), (1000, 1024), (37, 16388), (300, 8192), (129, 16384),
               # rows of 1-8 vectors (2-, 4- and 8-lane row groups), ragged row counts
               (1001, 4), (777, 8), (1000, 12), (513, 16), (299, 32),
               # 16-lane row groups in workgroups of 256 and 1024 threads
               (1500, 60), (3001, 64),
               # short misaligned rows (element-wise path, 8-64-lane groups)
               (1001, 7), (999, 33), (501, 101)]


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("shape", EDGE_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_edge_shapes_every_candidate(op, shape, dt):
    from paper_2512_22147_amd import mep

    m, n = shape
    ins = make_inputs(op, m, n, dt, seed=1000 + m + 7 * n)
    ref = oracle_outputs(op, ins, dt)
    scales = condition_scales(op, ins, dt)
    code = op_code(op)
    count = mep.mep_variant_count(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n)
    assert count >= 1
    for v in range(count):
        mep.mep_set_variant(code, v)
        got = gpu_outputs(op, ins, dt)
        assert_parity(op, got, ref, dt, what=f"{m}x{n} candidate {v}", scales=scales, dims=(m, n))


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("shape", [(2048, 4096), (513, 1027), (4000, 64), (3, 40000), (5001, 8), (3000, 12)],
                         ids=lambda s: f"{s[0]}x{s[1]}")
def test_integer_inputs_bit_exact(op, shape, dt):
    """Entries in {-1, 0, 1}: every partial sum is an integer below 2^24, so
    any summation order gives the exact result, in fp32 as in fp64."""
    m, n = shape
    ins = make_inputs(op, m, n, dt, seed=77 + m, kind="ternary")
    ref = oracle_outputs(op, ins, dt, alpha=1.5, beta=0.25)
    if op == "gemver":
        # Ahat is an integer matrix, x a multiple of 1/4, w of 1/8: exact while
        # every |partial sum| (bounded by |Ahat| |y| and |Ahat| |x|) and every
        # result stays below 2^24 in those units
        Ah = np.abs(ref["Ahat"])
        assert 4 * float(np.max(Ah.T @ np.abs(ins["y"].astype(np.float64)), initial=0)) < 2 ** 24
        assert 4 * float(np.max(Ah @ np.abs(ref["x"]), initial=0)) < 2 ** 24
        assert 8 * float(np.max(np.abs(ref["w"]), initial=0)) < 2 ** 24
    got = gpu_outputs(op, ins, dt, alpha=1.5, beta=0.25)
    for k, r in ref.items():
        assert np.array_equal(got[k].astype(np.float64), r), f"{op} {k} not exact"


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
def test_long_rows_use_column_panels(op, dt):
    """Rows longer than one on-chip row group: column panels (and for ATAX
    the two-pass path)."""
    n = 40000 if dt == np.float32 else 20000
    for m in (1, 67):
        ins = make_inputs(op, m, n, dt, seed=5 + m)
        assert_parity(op, gpu_outputs(op, ins, dt), oracle_outputs(op, ins, dt), dt,
                      what=f"{m}x{n}")


# Row lengths around the panel widths (the widest row group covers 32768 fp32
# or 16384 fp64 elements; GEMVER's first pass half that): just past one panel,
# three and more panels, odd lengths on the element-wise path.  The host cuts
# such rows into panels of equal width, a multiple of the vector width, and
# never leaves the last one empty.
PANEL_WIDTHS = {np.float32: [16388, 32772, 32769, 65540, 98308, 98307],
                np.float64: [8194, 16386, 16385, 40002, 49154]}


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
def test_equal_panels_every_candidate(op, dt):
    from paper_2512_22147_amd import mep

    code = op_code(op)
    for n in PANEL_WIDTHS[dt]:
        m = 37
        ins = make_inputs(op, m, n, dt, seed=300 + n % 1000)
        ref = oracle_outputs(op, ins, dt)
        scales = condition_scales(op, ins, dt)
        count = mep.mep_variant_count(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n)
        for v in range(count):
            mep.mep_set_variant(code, v)
            assert_parity(op, gpu_outputs(op, ins, dt), ref, dt, what=f"{m}x{n} candidate {v}", scales=scales,
                          dims=(m, n))
        mep.mep_set_variant(code, -1)


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
def test_misaligned_matrix_takes_elementwise_path(op, dt):
    import torch

    from paper_2512_22147_amd import mep

    m, n = 70, 516
    ins = make_inputs(op, m, n, dt, seed=9)
    ref = oracle_outputs(op, ins, dt)
    dev = torch.device("cuda:0")
    # A (and B) start one element past a 16-byte boundary
    raw = torch.empty(m * n + 1, dtype=torch.float32 if dt == np.float32 else torch.float64,
                      device=dev)
    A = raw[1:].view(m, n)
    A.copy_(torch.from_numpy(ins["A"]))
    assert A.data_ptr() % 16 != 0
    x = torch.from_numpy(ins.get("x", np.zeros(n, dt))).to(dev)
    if op == "matvec":
        got = {"y": mep.mep_matvec(A, x)}
    elif op == "matvec_t":
        got = {"z": mep.mep_matvec_t(A, torch.from_numpy(ins["w"]).to(dev))}
    elif op == "bicg":
        z, q = mep.mep_matvec_t(A, torch.from_numpy(ins["w"]).to(dev), p=x)
        got = {"z": z, "q": q}
    elif op == "ata_x":
        t = torch.empty(m, dtype=A.dtype, device=dev)
        got = {"y": mep.mep_ata_x(A, x, t=t), "t": t}
    elif op == "gemver":
        T = {k: torch.from_numpy(ins[k]).to(dev) for k in ("u1", "v1", "u2", "v2", "y", "z")}
        Ahat, xo, w = mep.mep_gemver(1.5, 1.2, A, T["u1"], T["v1"], T["u2"], T["v2"], T["y"], T["z"])
        got = {"Ahat": Ahat, "x": xo, "w": w}
    else:
        rawb = torch.empty_like(raw)
        Bm = rawb[1:].view(m, n)
        Bm.copy_(torch.from_numpy(ins["B"]))
        got = {"y": mep.mep_axpby_mv(1.5, A, 1.2, Bm, x)}
    torch.cuda.synchronize()
    assert_parity(op, {k: v.cpu().numpy() for k, v in got.items()}, ref, dt)


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
def test_empty_sizes(dt):
    """An empty sum is zero; zero-length outputs are left alone."""
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    tdt = torch.float32 if dt == np.float32 else torch.float64
    e = lambda *s: torch.empty(*s, dtype=tdt, device=dev)
    A0n = e(0, 5)
    Am0 = e(6, 0)
    assert mep.mep_matvec(Am0, e(0), y=torch.full((6,), 7.0, dtype=tdt, device=dev)).abs().sum() == 0
    assert mep.mep_matvec(A0n, e(5)).numel() == 0
    assert mep.mep_matvec_t(A0n, e(0), z=torch.full((5,), 7.0, dtype=tdt, device=dev)).abs().sum() == 0
    z, q = mep.mep_matvec_t(Am0, e(6), p=e(0), q=torch.full((6,), 7.0, dtype=tdt, device=dev))
    assert z.numel() == 0 and q.abs().sum() == 0
    assert mep.mep_ata_x(A0n, e(5), y=torch.full((5,), 7.0, dtype=tdt, device=dev)).abs().sum() == 0
    t = torch.full((6,), 7.0, dtype=tdt, device=dev)
    mep.mep_ata_x(Am0, e(0), t=t)
    assert t.abs().sum() == 0
    assert mep.mep_axpby_mv(1.0, Am0, 1.0, e(6, 0), e(0),
                            y=torch.full((6,), 7.0, dtype=tdt, device=dev)).abs().sum() == 0
    # GEMVER: no rows gives x = z; no columns gives w = 0
    z = torch.arange(5, dtype=tdt, device=dev) + 0.5
    _, xo, w = mep.mep_gemver(1.5, 1.2, A0n, e(0), e(5), e(0), e(5), e(0), z,
                              x=torch.full((5,), 7.0, dtype=tdt, device=dev))
    assert torch.equal(xo, z) and w.numel() == 0
    _, xo, w = mep.mep_gemver(1.5, 1.2, Am0, e(6), e(0), e(6), e(0), e(6), e(0),
                              w=torch.full((6,), 7.0, dtype=tdt, device=dev))
    assert xo.numel() == 0 and w.abs().sum() == 0
    torch.cuda.synchronize()


@pytest.mark.parametrize("op", OPS)
def test_guards_and_reproducibility(op):
    """Nothing is written past the outputs or the workspace, and two runs give
    bitwise-identical results (fixed-order reductions)."""
    import torch

    from paper_2512_22147_amd import mep

    dt = np.float32
    m, n = 3000, 4100
    ins = make_inputs(op, m, n, dt, seed=31)
    dev = torch.device("cuda:0")
    T = {k: torch.from_numpy(v).to(dev) for k, v in ins.items()}
    code = op_code(op)
    need = mep.mep_workspace_bytes(code, mep.MEP_F32, m, n)
    G = 4096
    guard = 0x5A
    ws_all = torch.full((need + G,), guard, dtype=torch.uint8, device=dev)
    ws = ws_all[:need] if need else None
    out_len = {"matvec": m, "matvec_t": n, "bicg": n, "ata_x": n, "axpby_mv": m, "gemver": n}[op]
    sentinel = 12345.0
    runs = []
    for _ in range(2):
        o = torch.full((out_len + G,), sentinel, dtype=torch.float32, device=dev)
        q = torch.full((m + G,), sentinel, dtype=torch.float32, device=dev)
        hat = torch.full((m * n + G,), sentinel, dtype=torch.float32, device=dev)
        y = o[:out_len]
        if op == "matvec":
            mep.mep_matvec(T["A"], T["x"], y=y, ws=ws)
        elif op == "matvec_t":
            mep.mep_matvec_t(T["A"], T["w"], z=y, ws=ws)
        elif op == "bicg":
            mep.mep_matvec_t(T["A"], T["w"], z=y, p=T["x"], q=q[:m], ws=ws)
        elif op == "ata_x":
            mep.mep_ata_x(T["A"], T["x"], y=y, t=q[:m], ws=ws)
        elif op == "gemver":
            mep.mep_gemver(1.5, 1.2, T["A"], T["u1"], T["v1"], T["u2"], T["v2"], T["y"], T["z"],
                           x=y, w=q[:m], Ahat=hat[:m * n].view(m, n), ws=ws)
        else:
            mep.mep_axpby_mv(1.5, T["A"], 1.2, T["B"], T["x"], y=y, ws=ws)
        torch.cuda.synchronize()
        assert bool((o[out_len:] == sentinel).all()), "write past the output"
        assert bool((q[m:] == sentinel).all()), "write past the second output"
        assert bool((hat[m * n:] == sentinel).all()), "write past the updated matrix"
        assert bool((ws_all[need:] == guard).all()), "write past the workspace"
        runs.append(torch.cat([y, q[:m], hat[:m * n] if op == "gemver" else q[:0]]).cpu().numpy())
    assert np.array_equal(runs[0].view(np.uint32), runs[1].view(np.uint32))


def test_harness_on_gpu():
    """mep_time_trimmed (Eq. 3), profiling events and the copy probe."""
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    m, n = 2048, 2048
    A = torch.randn(m, n, device=dev)
    x = torch.randn(n, device=dev)
    y = torch.empty(n, device=dev)
    flush = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
    call = mep.make_call(mep.MEP_OP_ATA_X, A, in0=x, out0=y, flush_buf=flush)
    mean, samples = mep.mep_time_trimmed(call, warmup=2, R=9, k=2, inner=3, flush=True)
    assert len(samples) == 9 and all(s > 0 for s in samples)
    assert mean == pytest.approx(mep.mep_trimmed_mean(samples, 2), rel=1e-12)
    mep.mep_profile_begin(8)
    for _ in range(5):
        mep.mep_run(call)
    tot, cnt = mep.mep_profile_end()
    assert cnt == 5 and tot > 0
    # a GEMVER call records both of its streaming passes
    u = torch.randn(m, device=dev)
    v = torch.randn(n, device=dev)
    g = mep.make_call(mep.MEP_OP_GEMVER, A, in0=u, in1=v, in2=u, in3=v, in4=u, in5=v,
                      out0=torch.empty(n, device=dev), out1=torch.empty(m, device=dev),
                      out2=torch.empty_like(A), alpha=1.5, beta=1.2)
    mep.mep_profile_begin(8)
    for _ in range(3):
        mep.mep_run(g)
    samples, tot, cnt = mep.mep_profile_end_samples(8)
    assert cnt == 6 and len(samples) == 6 and all(t > 0 for t in samples)
    assert tot == pytest.approx(sum(samples), rel=1e-9)
    # sampled stamping: groups of GEMVER's two launches, every third group
    # (7 calls = 14 launches -> launches 0, 1, 6, 7, 12, 13)
    mep.mep_profile_begin_sampled(16, 2, 3)
    for _ in range(7):
        mep.mep_run(g)
    samples, tot, cnt = mep.mep_profile_end_samples(16)
    assert cnt == 6 and len(samples) == 6 and all(t > 0 for t in samples)
    mep.mep_profile_begin(4)
    with pytest.raises(mep.MepError):
        mep.mep_profile_end_samples(-1)
    src = torch.arange(1 << 20, dtype=torch.int32, device=dev)
    dst = torch.zeros_like(src)
    mep.mep_stream_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


FULL = [("ata_x_1024", "f32"), ("bicg_4096", "f32"), ("axpby_mv_8192", "f32"),
        ("ata_x_16384", "f32"), ("ata_x_16384", "f64"), ("matvec_t_1m_x_64", "f32"),
        ("gemver_16384", "f32")]


@pytest.mark.parametrize("name,dts", FULL, ids=[f"{a}-{b}" for a, b in FULL])
def test_full_size_workloads(name, dts):
    """The benchmark workloads at full size, default kernel candidate (the
    launch configuration bench.py times), every output element against the
    oracle; the headline workload also run twice for bitwise equality."""
    from paper_2512_22147_amd import datagen

    w = datagen.WORKLOADS[name]
    dt = np.float32 if dts == "f32" else np.float64
    raw = datagen.make_inputs(w, dt)
    op = w.op
    if op == "bicg":
        ins = {"A": raw["A"], "x": raw["p"], "w": raw["r"]}
    else:
        ins = dict(raw)
    ref = oracle_outputs(op, ins, dt, alpha=w.alpha or 1.5, beta=w.beta or 1.2)
    scales = condition_scales(op, ins, dt, alpha=w.alpha or 1.5, beta=w.beta or 1.2)
    got = gpu_outputs(op, ins, dt, alpha=w.alpha or 1.5, beta=w.beta or 1.2)
    assert_parity(op, got, ref, dt, what=name, scales=scales, dims=ins["A"].shape)
    if name == "ata_x_16384":
        again = gpu_outputs(op, ins, dt)
        for k in got:
            assert np.array_equal(got[k], again[k]), f"{k} differs between runs"


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("shape", [(3000, 4100), (67, 40000), (1000, 1024)],
                         ids=lambda s: f"{s[0]}x{s[1]}")
def test_gemver_in_place(shape, dt):
    """Ahat = A (the in-place update) gives bitwise the out-of-place results."""
    import torch

    from paper_2512_22147_amd import mep

    m, n = shape
    ins = make_inputs("gemver", m, n, dt, seed=606 + m)
    dev = torch.device("cuda:0")
    T = {k: torch.from_numpy(v).to(dev) for k, v in ins.items()}
    vecs = [T[k] for k in ("u1", "v1", "u2", "v2", "y", "z")]
    Ahat, x, w = mep.mep_gemver(1.5, 1.2, T["A"], *vecs)
    A2 = T["A"].clone()
    Ahat2, x2, w2 = mep.mep_gemver(1.5, 1.2, A2, *vecs, Ahat=A2)
    torch.cuda.synchronize()
    assert Ahat2.data_ptr() == A2.data_ptr()
    assert torch.equal(Ahat, A2) and torch.equal(x, x2) and torch.equal(w, w2)
    assert_parity("gemver", {"Ahat": A2.cpu().numpy(), "x": x2.cpu().numpy(), "w": w2.cpu().numpy()},
                  oracle_outputs("gemver", ins, dt, alpha=1.5, beta=1.2), dt)


@pytest.mark.parametrize("op,shape", [("ata_x", (3000, 4096)), ("matvec_t", (100000, 64)),
                                      ("axpby_mv", (2000, 2048)), ("bicg", (1024, 1024)),
                                      ("gemver", (1000, 2048))])
def test_select_variant_eqs_3_to_5(op, shape):
    """The Sec. 3.2 selection over the candidate kernels: every candidate
    passes FE against the baseline, the winner is the argmin of the Eq. 3
    means (as the oracle's selection rule computes it from the same list),
    and once applied the operation still matches the oracle."""
    import torch

    import oracle
    from paper_2512_22147_amd import mep

    m, n = shape
    dt = np.float32
    ins = make_inputs(op, m, n, dt, seed=404)
    dev = torch.device("cuda:0")
    T = {k: torch.from_numpy(v).to(dev) for k, v in ins.items()}
    code = op_code(op)
    out0 = torch.empty(m if op in ("matvec", "axpby_mv") else n, device=dev)
    out1 = torch.empty(m, device=dev) if op in ("bicg", "ata_x", "gemver") else None
    kw = dict(out0=out0, out1=out1)
    if op == "gemver":
        call = mep.make_call(code, T["A"], in0=T["u1"], in1=T["v1"], in2=T["u2"], in3=T["v2"],
                             in4=T["y"], in5=T["z"], out2=torch.empty_like(T["A"]), alpha=1.5,
                             beta=1.2, **kw)
    elif op == "ata_x":
        call = mep.make_call(code, T["A"], in0=T["x"], **kw)
    elif op == "bicg":
        call = mep.make_call(code, T["A"], in0=T["w"], in1=T["x"], **kw)
    elif op == "matvec_t":
        call = mep.make_call(code, T["A"], in0=T["w"], out0=out0)
    else:
        call = mep.make_call(code, T["A"], in0=T["x"], B=T["B"], alpha=1.5, beta=1.2, out0=out0)
    # warm timing (flush=False) with a flush buffer: the caches are cleared
    # once before each candidate; a buffer of a size that is not a multiple
    # of 16 bytes is refused before anything runs
    fb = torch.empty(16 << 20, dtype=torch.uint8, device=dev)
    call.flush_buf, call.flush_bytes = fb.data_ptr(), fb.numel() - 8
    with pytest.raises(mep.MepError):
        mep.mep_select_variant(call, warmup=1, R=7, k=2, tol=1e-4, apply=True)
    call.flush_bytes = fb.numel()
    best, res = mep.mep_select_variant(call, warmup=1, R=7, k=2, tol=1e-4, apply=True)
    assert len(res) == mep.mep_variant_count(code, mep.MEP_F32, m, n)
    assert all(ok for _, _, ok in res), res
    assert best == oracle.select_next([(i, t, ok) for i, (t, _, ok) in enumerate(res)])
    got = gpu_outputs(op, ins, dt)
    assert_parity(op, got, oracle_outputs(op, ins, dt), dt, what=f"selected candidate {best}")


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", ["matvec_t", "bicg", "ata_x", "gemver"])
@pytest.mark.parametrize("shape", [(200000, 64), (150001, 7), (300000, 128), (70000, 1)],
                         ids=lambda s: f"{s[0]}x{s[1]}")
def test_narrow_outputs_split_reduce(op, shape, dt):
    """Many rows, few columns: hundreds of partial rows of a narrow output
    and the element-wise path for odd widths.  Every candidate against the
    oracle, and three runs bit for bit alike."""
    from paper_2512_22147_amd import mep

    m, n = shape
    ins = make_inputs(op, m, n, dt, seed=4242 + n)
    ref = oracle_outputs(op, ins, dt)
    code = op_code(op)
    count = mep.mep_variant_count(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n)
    for v in range(count):
        mep.mep_set_variant(code, v)
        runs = [gpu_outputs(op, ins, dt) for _ in range(3)]
        assert_parity(op, runs[0], ref, dt, what=f"{m}x{n} candidate {v}")
        for k in ref:
            assert runs[0][k].tobytes() == runs[1][k].tobytes() == runs[2][k].tobytes(), \
                f"{op} {k} candidate {v} differs between runs"


# One shape per range of the default-shape rule (rows of 1-8193 vectors,
# both sides of every split point), with enough rows that every workgroup
# loops over several batches: the defaults of every op against the oracle.
DEFAULT_RULE_SHAPES = [(100003, 4), (60001, 8), (40000, 12), (30001, 16), (20000, 32),
                       (50001, 7), (20001, 33), (10001, 101), (3001, 1001),
                       (2600, 2052), (1800, 3072), (1800, 3076), (1400, 4100), (1000, 6148),
                       (800, 8196), (500, 12292), (400, 16388), (300, 24580)]


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("shape", DEFAULT_RULE_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_default_shapes_across_row_lengths(op, shape):
    from paper_2512_22147_amd import mep

    m, n = shape
    for dt in DTYPES:
        if dt == np.float64 and n % 2:
            continue
        ins = make_inputs(op, m, n, dt, seed=5000 + m + n)
        ref = oracle_outputs(op, ins, dt)
        code = op_code(op)
        info = mep.mep_variant_info(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n, 0)
        got = gpu_outputs(op, ins, dt)
        assert_parity(op, got, ref, dt, what=f"{m}x{n} default ({info})")


def _random_cases(count=72, seed=2026):
    """Seeded random shapes over the whole planning space: row lengths from 1
    to ~70000 elements (narrow groups, vector and element-wise paths, column
    panels), 1 to ~20000 rows, every op and both dtypes; sized so that the
    oracle finishes each in well under a second."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        n = int(np.exp(rng.uniform(0, np.log(70000))))
        m = int(np.exp(rng.uniform(0, np.log(20000))))
        if m * n > 6_000_000:
            continue
        op = OPS[int(rng.integers(len(OPS)))]
        dt = DTYPES[int(rng.integers(2))]
        cases.append((op, m, n, dt))
    return cases


RANDOM_CASES = _random_cases()


def _random_streamed_cases(count=24, seed=99):
    """Seeded random shapes of matrices too large for the Infinity Cache
    (150-400 MB), where the default shapes differ from the cache-resident
    ones (narrowed grids, other batch depths): row lengths of 1 to ~40000
    elements, every op and both dtypes."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        n = int(np.exp(rng.uniform(0, np.log(40000))))
        dt = DTYPES[int(rng.integers(2))]
        es = np.dtype(dt).itemsize
        m = max(1, int(rng.uniform(150e6, 400e6) / (n * es)))
        op = OPS[int(rng.integers(len(OPS)))]
        if op == "gemver" and m * n * es > 250e6:
            continue
        cases.append((op, m, n, dt))
    return cases


RANDOM_STREAMED_CASES = _random_streamed_cases()


@pytest.mark.parametrize("case", range(len(RANDOM_CASES)))
def test_random_shapes(case):
    op, m, n, dt = RANDOM_CASES[case]
    ins = make_inputs(op, m, n, dt, seed=7000 + case)
    ref = oracle_outputs(op, ins, dt)
    got = gpu_outputs(op, ins, dt)
    assert_parity(op, got, ref, dt, what=f"case {case}: {op} {m}x{n} {np.dtype(dt).name}",
                  scales=condition_scales(op, ins, dt), dims=(m, n))


@pytest.mark.parametrize("case", range(len(RANDOM_STREAMED_CASES)))
def test_random_streamed_shapes(case):
    op, m, n, dt = RANDOM_STREAMED_CASES[case]
    ins = make_inputs(op, m, n, dt, seed=9100 + case)
    ref = oracle_outputs(op, ins, dt)
    got = gpu_outputs(op, ins, dt)
    assert_parity(op, got, ref, dt, what=f"streamed case {case}: {op} {m}x{n} {np.dtype(dt).name}")


@pytest.mark.parametrize("nbytes", [16, 48, (128 << 10) + 16, (3 << 20) + 48, 64 << 20, (1 << 30) + 4096])
def test_stream_copy_sizes(nbytes):
    """The copy probe copies every byte, ragged last row included, and
    writes nothing past dst."""
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(nbytes % 1000)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device=dev, generator=g)
    guard = 4096
    dst_all = torch.full((nbytes + guard,), 0xA5, dtype=torch.uint8, device=dev)
    mep.mep_stream_copy(src, dst_all[:nbytes])
    torch.cuda.synchronize()
    assert torch.equal(src, dst_all[:nbytes])
    assert bool((dst_all[nbytes:] == 0xA5).all())


@pytest.mark.parametrize("dt", DTYPES, ids=["f32", "f64"])
@pytest.mark.parametrize("op", OPS)
def test_small_rows_and_columns(op, dt):
    """Rows and columns of A (and B) scaled by 2^-20 (exactly): their outputs
    have error scales far below max|ref|, where the normwise check is blind
    and the condition-scaled bound is what holds them."""
    from paper_2512_22147_amd import mep

    m, n = 1500, 2052
    ins = make_inputs(op, m, n, dt, seed=4242)
    for name in ("A", "B"):
        if name in ins:
            ins[name][::7, :] *= dt(2.0**-20)
            ins[name][:, 3::11] *= dt(2.0**-20)
    ref = oracle_outputs(op, ins, dt)
    scales = condition_scales(op, ins, dt)
    code = op_code(op)
    for v in range(mep.mep_variant_count(code, mep.MEP_F32 if dt == np.float32 else mep.MEP_F64, m, n)):
        mep.mep_set_variant(code, v)
        got = gpu_outputs(op, ins, dt)
        assert_parity(op, got, ref, dt, what=f"{m}x{n} candidate {v}", scales=scales, dims=(m, n))


ROTATED_CASES = [(np.float32, 1, 11300), (np.float32, 385, 12292), (np.float32, 2731, 12300),
                 (np.float32, 5000, 16384), (np.float64, 1, 12000), (np.float64, 211, 12300),
                 (np.float64, 1500, 12300), (np.float64, 3000, 16384)]


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("case", ROTATED_CASES,
                         ids=lambda c: f"{'f32' if c[0] == np.float32 else 'f64'}-{c[1]}x{c[2]}")
def test_rotated_block_map(op, case):
    """The rotated row-block map (fp32 rows of 2817-4096 vectors, fp64 rows
    of 5633-8192): one row, a second round holding a single block, and
    several rounds with a ragged last one, including streamed matrices (the
    default shape for fp32 y = A x, A^T w, BICG and ATAX, and for fp64
    ATAX); the same bits on a second run."""
    from paper_2512_22147_amd import mep

    dt, m, n = case
    code = op_code(op)
    dcode = mep.MEP_F32 if dt == np.float32 else mep.MEP_F64
    infos = [mep.mep_variant_info(code, dcode, m, n, v) for v in range(mep.mep_variant_count(code, dcode, m, n))]
    rot = [v for v, s in enumerate(infos) if "rotated" in s]
    if not rot:
        pytest.skip(f"no rotated candidate for {op} at {m}x{n}")
    streamed = m * n * np.dtype(dt).itemsize > (128 << 20)
    if streamed and (op == "ata_x" or (dt == np.float32 and op in ("matvec", "matvec_t", "bicg"))):
        assert rot[0] == 0, "a streamed row of this length takes the rotated map by default"
    ins = make_inputs(op, m, n, dt, seed=7000 + m)
    ref = oracle_outputs(op, ins, dt)
    scales = condition_scales(op, ins, dt)
    try:
        mep.mep_set_variant(code, rot[0])
        got = gpu_outputs(op, ins, dt)
        again = gpu_outputs(op, ins, dt)
    finally:
        mep.mep_set_variant(code, -1)
    assert_parity(op, got, ref, dt, what=f"{m}x{n} {infos[rot[0]]}", scales=scales, dims=(m, n))
    for k in got:
        assert got[k].tobytes() == again[k].tobytes(), f"{k} differs between two runs"
