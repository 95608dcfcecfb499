"""The operations only enqueue kernels (no allocation, no memset, no host
synchronization), so a caller can capture them into a HIP graph.  Each graph
is replayed several times, with eager work and synchronizations in between,
and every replay must equal the eager result bit for bit."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _calls(torch, mep, dev, dt):
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    r = lambda *s: torch.rand(*s, generator=g, device=dev, dtype=dt) * 2 - 1
    m, n = 3000, 4100
    A, B = r(m, n), r(m, n)
    x, w, p = r(n), r(m), r(n)
    out = {}
    calls = []
    ws = lambda op: torch.empty(max(mep.mep_workspace_bytes(op, mep.dtype_code(dt), m, n), 1),
                                dtype=torch.uint8, device=dev)
    out["ata_y"] = torch.empty(n, device=dev, dtype=dt)
    calls.append(mep.make_call(mep.MEP_OP_ATA_X, A, in0=x, out0=out["ata_y"], ws=ws(mep.MEP_OP_ATA_X)))
    out["bicg_s"], out["bicg_q"] = torch.empty(n, device=dev, dtype=dt), torch.empty(m, device=dev, dtype=dt)
    calls.append(mep.make_call(mep.MEP_OP_BICG, A, in0=w, in1=p, out0=out["bicg_s"], out1=out["bicg_q"],
                               ws=ws(mep.MEP_OP_BICG)))
    out["gesummv"] = torch.empty(m, device=dev, dtype=dt)
    calls.append(mep.make_call(mep.MEP_OP_AXPBY_MV, A, in0=x, B=B, alpha=1.5, beta=1.2, out0=out["gesummv"],
                               ws=ws(mep.MEP_OP_AXPBY_MV)))
    out["gemver_x"], out["gemver_w"] = torch.empty(n, device=dev, dtype=dt), torch.empty(m, device=dev, dtype=dt)
    out["gemver_Ahat"] = torch.empty_like(A)
    calls.append(mep.make_call(mep.MEP_OP_GEMVER, A, in0=w, in1=x, in2=w, in3=p, in4=w, in5=x,
                               out0=out["gemver_x"], out1=out["gemver_w"], out2=out["gemver_Ahat"],
                               alpha=1.5, beta=1.2, ws=ws(mep.MEP_OP_GEMVER)))
    v = r(1 << 22)
    out["sum"] = torch.empty(1, device=dev, dtype=dt)
    calls.append(mep.make_call(mep.MEP_OP_REDUCE_SUM, v, out0=out["sum"]))
    out["add"] = torch.empty_like(v)
    calls.append(mep.make_call(mep.MEP_OP_VECTOR_ADD, v, in1=v, out0=out["add"]))
    keep = (A, B, x, w, p, v)
    return calls, out, keep


@pytest.mark.parametrize("dt", ["f32", "f64"])
def test_operations_replay_from_a_captured_graph(dt):
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    tdt = torch.float32 if dt == "f32" else torch.float64
    s = torch.cuda.Stream()
    calls, out, keep = _calls(torch, mep, dev, tdt)
    for c in calls:
        c.stream = s.cuda_stream
    with torch.cuda.stream(s):
        for c in calls:
            mep.mep_run(c)
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in out.items()}
    for v in out.values():
        v.fill_(float("nan"))
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        for c in calls:
            mep.mep_run(c)
    for rep in range(4):
        # eager work of the program's own between the replays
        junk = torch.randn(1 << 20, device=dev).sum()
        torch.cuda.synchronize()
        for v in out.values():
            v.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for k, v in out.items():
            assert torch.equal(v, eager[k]), f"replay {rep}: {k} differs from the eager result"
        del junk
    del keep
