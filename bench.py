#!/usr/bin/env python3
"""Benchmark of the dense matrix-vector MEPs on one MI355X (gfx950).

Default workload: the fused y = A^T (A x) over a 16384 x 16384 fp32 matrix
(uniform[-1,1) from seed 3).  A step is one call of the operation: for ATAX
the matrix-streaming kernel (row dot and transposed accumulation in one read
of A) plus the fixed-order column reduction.  Inputs are resident in HBM
before timing starts; W warm-up steps, then exactly K timed steps between two
device synchronizations.  One JSON line is printed:

* value        -- whole-step throughput: algorithmic bytes (every input once,
                  every output once) per second
* roofline     -- the dominant kernel's algorithmic bytes per launch divided by
                  its average duration, from event pairs stamped by the
                  launches of every 8th step of the timed region, on the
                  kernel's own stream; traffic is the calibrated rocprofv3 HBM
                  byte count per launch
* eq3          -- the MEP timing rule of Eq. 3 on the GPU: 3 warm-up calls,
                  R = 30 samples, each after a 1 GiB cache flush, trimmed
                  mean with the k = 3 fastest and slowest dropped
* cpu_baseline -- the CPU oracle, as it stands, on the host cores

Other workloads (--workload): ata_x_1024, bicg_4096, axpby_mv_8192,
matvec_t_1m_x_64, gemver_16384, reduce_sum_256m, vector_add_256m.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HEADLINE = "ata_x_16384"
# the other benchmark configurations (parity cases), timed beside the headline:
# whole steps (all kernels of the operation) on resident inputs, the default shape
OTHER_CONFIGS = [("ata_x_1024", "f32"), ("bicg_4096", "f32"), ("axpby_mv_8192", "f32"),
                 ("matvec_t_1m_x_64", "f32")]
HEADLINE_METRIC = "achieved HBM GB/s (and % of MI355X peak) for y=Aᵀ(Ax), fp32 16384²"
PEAK_GBS = 8000.0
KERNEL_SOURCE = "paper_2512_22147_amd/csrc/mep_kernels.hpp"
VECTOR_KERNEL_SOURCE = "paper_2512_22147_amd/csrc/mep_vector_kernels.hpp"


def kernel_source_hash(workload: str = "") -> str:
    """Stamp of the source the workload's dominant kernel is built from."""
    vector = workload.startswith(("reduce_sum", "vector_add"))
    h = hashlib.sha256()
    for rel in ((KERNEL_SOURCE, VECTOR_KERNEL_SOURCE) if vector else (KERNEL_SOURCE,)):
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, dtype: str, config: str):
    """HBM bytes (fetched + written) per launch of the dominant kernel from the
    committed rocprofv3 counter summary; None when the summary is absent or was
    taken on another kernel source or another configuration."""
    path = os.path.join(ROOT, "profiles", f"{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    if not m or m.group(1) != kernel_source_hash(workload):
        return None
    m = re.search(rf"config_{dtype}:\s*(.+)", text)
    if not m or m.group(1).strip() != config:
        return None
    m = re.search(rf"traffic_bytes_per_launch_{dtype}:\s*([0-9.eE+]+)", text)
    return float(m.group(1)) if m else None


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--dtype", choices=["f32", "f64"], default="f32")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-f64", action="store_true", help="skip the fp64 secondary measurement")
    ap.add_argument("--probe-copy", action="store_true",
                    help="also run the 1 GiB streaming-copy probe (counter calibration)")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the HBM ceiling probe (a read-sum of as many bytes as the workload streams)")
    ap.add_argument("--variant", type=int, default=-1, help="kernel candidate (Eqs. 4-5); -1 default")
    ap.add_argument("--select", action="store_true",
                    help="also run one round of candidate selection (Eqs. 3-5, cold cache) and report "
                         "the chosen shape's standalone speedup over the default (Sec. 4.1.4)")
    ap.add_argument("--no-eq3", action="store_true",
                    help="skip the Eq. 3 cold-cache timing (R = 30, k = 3, 1 GiB flush per sample)")
    ap.add_argument("--probe-floor", action="store_true",
                    help="also time back-to-back launches of a 16-byte copy (the launch floor)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the step timing of the other benchmark configurations (reported beside "
                         "the headline as other_configs)")
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


OPS = {
    # workload op -> (mep op code attribute, dominant kernel, description)
    "ata_x": ("MEP_OP_ATA_X", "k_stream (ATAX mode)", "y = A^T (A x)"),
    "bicg": ("MEP_OP_BICG", "k_stream (BICG mode)", "q = A p and s = A^T r"),
    "axpby_mv": ("MEP_OP_AXPBY_MV", "k_stream (AXPBY mode)", "y = alpha A x + beta B x"),
    "matvec_t": ("MEP_OP_MATVEC_T", "k_stream (A^T w mode)", "z = A^T w"),
    "reduce_sum": ("MEP_OP_REDUCE_SUM", "k_reduce_sum", "s = sum x"),
    "vector_add": ("MEP_OP_VECTOR_ADD", "k_vector_add_buf", "c = a + b"),
    "gemver": ("MEP_OP_GEMVER", "k_stream (GEMVER pass 1: Ahat stored, Ahat^T y)",
               "GEMVER Ahat = A + u1 v1^T + u2 v2^T, x = beta Ahat^T y + z, w = alpha Ahat x"),
}


def setup(workload: str, dtype: str):
    """Device inputs, one step as a closure, and the byte counts."""
    import numpy as np
    import torch

    from paper_2512_22147_amd import datagen, mep

    w = datagen.WORKLOADS[workload]
    npdt = np.float32 if dtype == "f32" else np.float64
    es = np.dtype(npdt).itemsize
    log(f"[bench] generating {workload} {dtype}")
    host = datagen.make_inputs(w, npdt)
    dev = torch.device("cuda:0")
    d = {k: torch.from_numpy(v).to(dev) for k, v in host.items()}
    torch.cuda.synchronize()
    m, n = w.m, w.n
    code = getattr(mep, OPS[w.op][0])
    tdt = d[next(iter(d))].dtype
    need = mep.mep_workspace_bytes(code, mep.dtype_code(tdt), m, n)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    # one prebuilt mep_call_t per workload: a step is a single mep_run call
    if w.op == "ata_x":
        y = torch.empty(n, dtype=tdt, device=dev)
        call = mep.make_call(code, d["A"], in0=d["x"], out0=y, ws=ws)
        outs = lambda: {"y": y}
        alg_step, alg_kernel = (m * n + 2 * n) * es, (m * n + n) * es
    elif w.op == "bicg":
        z = torch.empty(n, dtype=tdt, device=dev)
        q = torch.empty(m, dtype=tdt, device=dev)
        call = mep.make_call(code, d["A"], in0=d["r"], in1=d["p"], out0=z, out1=q, ws=ws)
        outs = lambda: {"q": q, "s": z}
        alg_step, alg_kernel = (m * n + 2 * n + 2 * m) * es, (m * n + n + 2 * m) * es
    elif w.op == "axpby_mv":
        y = torch.empty(m, dtype=tdt, device=dev)
        call = mep.make_call(code, d["A"], in0=d["x"], B=d["B"], alpha=w.alpha, beta=w.beta, out0=y, ws=ws)
        outs = lambda: {"y": y}
        alg_step = alg_kernel = (2 * m * n + n + m) * es
    elif w.op == "matvec_t":
        z = torch.empty(n, dtype=tdt, device=dev)
        call = mep.make_call(code, d["A"], in0=d["w"], out0=z, ws=ws)
        outs = lambda: {"z": z}
        alg_step, alg_kernel = (m * n + m + n) * es, (m * n + m) * es
    elif w.op == "reduce_sum":
        sv = torch.empty(1, dtype=tdt, device=dev)
        call = mep.make_call(code, d["x"], out0=sv, ws=ws)
        outs = lambda: {"s": sv}
        alg_step, alg_kernel = (n + 1) * es, n * es
    elif w.op == "gemver":
        x = torch.empty(n, dtype=tdt, device=dev)
        wv = torch.empty(m, dtype=tdt, device=dev)
        Ahat = torch.empty_like(d["A"])
        call = mep.make_call(code, d["A"], in0=d["u1"], in1=d["v1"], in2=d["u2"], in3=d["v2"],
                             in4=d["y"], in5=d["z"], out0=x, out1=wv, out2=Ahat, alpha=w.alpha,
                             beta=w.beta, ws=ws)
        outs = lambda: {"Ahat": Ahat, "x": x, "w": wv}
        # inputs once, outputs once, and the second pass's read of Ahat and x
        # (w needs the whole x, which needs the whole of Ahat)
        alg_step = (3 * m * n + 4 * m + 5 * n) * es
        alg_kernel = (2 * m * n + 3 * m + 2 * n) * es
        kernels = [(OPS["gemver"][1], alg_kernel),
                   ("k_stream (GEMVER pass 2: w = alpha Ahat x)", (m * n + m + n) * es)]
    else:
        c = torch.empty(n, dtype=tdt, device=dev)
        call = mep.make_call(code, d["a"], in1=d["b"], out0=c)
        outs = lambda: {"c": c}
        alg_step = alg_kernel = 3 * n * es
    if w.op != "gemver":
        kernels = [(OPS[w.op][1], alg_kernel)]
    step = lambda: mep.mep_run(call)
    return dict(w=w, code=code, step=step, outs=outs, alg_step=alg_step, alg_kernel=alg_kernel,
                kernels=kernels, host=host, dev=d, ws=ws, m=m, n=n, tdt=tdt, call=call)


def oracle_outputs(w, host, dtype):
    import numpy as np

    import oracle

    if w.op == "ata_x":
        return {"y": oracle.ata_x(host["A"], host["x"])[0]}
    if w.op == "bicg":
        q, s = oracle.bicg(host["A"], host["p"], host["r"])
        return {"q": q, "s": s}
    if w.op == "axpby_mv":
        npdt = np.float32 if dtype == "f32" else np.float64
        return {"y": oracle.axpby_mv(oracle.elem_scalar(w.alpha, npdt), host["A"],
                                     oracle.elem_scalar(w.beta, npdt), host["B"], host["x"])}
    if w.op == "matvec_t":
        return {"z": oracle.matvec_t(host["A"], host["w"])}
    if w.op == "reduce_sum":
        return {"s": np.array([oracle.reduce_sum(host["x"])])}
    if w.op == "gemver":
        npdt = np.float32 if dtype == "f32" else np.float64
        Ahat, x, wv = oracle.gemver(oracle.elem_scalar(w.alpha, npdt), oracle.elem_scalar(w.beta, npdt),
                                    host["A"], host["u1"], host["v1"], host["u2"], host["v2"],
                                    host["y"], host["z"])
        return {"Ahat": Ahat, "x": x, "w": wv}
    return {"c": oracle.vector_add(host["a"], host["b"])}


# Eq. 3 as the MEP harness applies it (Sec. 3.2, R = 30 and k = 3 from Sec. 4.1.3;
# three untimed warm-up calls): each sample is one call (or `inner` back-to-back
# calls when one call is shorter than T_min) timed by events on the call's stream,
# after a 1 GiB write that evicts every operand from the caches.
EQ3 = {"warmup": 3, "R": 30, "k": 3, "flush_bytes": 1 << 30}


def eq3_timing(S, ms_step):
    import math

    import torch

    from paper_2512_22147_amd import mep

    flush = torch.empty(EQ3["flush_bytes"], dtype=torch.uint8, device=torch.device("cuda:0"))
    call = S["call"]
    call.flush_buf, call.flush_bytes = flush.data_ptr(), EQ3["flush_bytes"]
    inner = max(1, math.ceil(T_MIN_MS / ms_step))
    mean_ms, samples = mep.mep_time_trimmed(call, warmup=EQ3["warmup"], R=EQ3["R"], k=EQ3["k"],
                                            inner=inner, flush=True)
    call.flush_buf, call.flush_bytes = None, 0
    del flush
    gbs = S["alg_step"] / (mean_ms * 1e-3) / 1e9
    return {**EQ3, "inner": inner, "trimmed_mean_ms": round(mean_ms, 5),
            "min_ms": round(min(samples), 5), "max_ms": round(max(samples), 5),
            "gbs": round(gbs, 1), "frac": round(gbs / PEAK_GBS, 4)}


def select_round(workload: str, dtype: str):
    """One round of the paper's loop over the library's candidate shapes: FE
    against the baseline (candidate 0), Eq. 3 timing with a cache flush per
    sample, argmin (Eqs. 4-5); the speedup counts only an FE-passing winner."""
    import torch

    from paper_2512_22147_amd import mep, report

    S = setup(workload, dtype)
    flush = torch.empty(EQ3["flush_bytes"], dtype=torch.uint8, device=torch.device("cuda:0"))
    call = S["call"]
    call.flush_buf, call.flush_bytes = flush.data_ptr(), EQ3["flush_bytes"]
    tol = 1e-4 if dtype == "f32" else 1e-12
    best, res = mep.mep_select_variant(call, warmup=EQ3["warmup"], R=EQ3["R"], k=EQ3["k"], flush=True,
                                       tol=tol, apply=False)
    dt = mep.dtype_code(S["tdt"])
    per = [{"candidate": i, "config": mep.mep_variant_info(S["code"], dt, S["m"], S["n"], i),
            "trimmed_mean_ms": None if r[0] != r[0] else round(r[0], 5), "fe_err": float(f"{r[1]:.3g}"),
            "fe_pass": r[2]} for i, r in enumerate(res)]
    out = {"workload": workload, "dtype": dtype, "per_candidate": per,
           "candidates": len(res), "fe_passed": sum(1 for r in res if r[2]), "best": best,
           "best_config": mep.mep_variant_info(S["code"], dt, S["m"], S["n"], max(best, 0)),
           "baseline_config": mep.mep_variant_info(S["code"], dt, S["m"], S["n"], 0),
           "baseline_ms": round(res[0][0], 5), "best_ms": round(res[best][0], 5) if best >= 0 else None,
           "standalone_speedup": report.selection_speedup(res, best)}
    log(f"[bench] selection: candidate {best} of {len(res)}, speedup {out['standalone_speedup']}")
    del S, flush
    torch.cuda.empty_cache()
    return out


PROFILE_EVERY = 8


def graph_step_ms(S, steps: int) -> float:
    """Device time per step with the host out of the way: the K steps are
    captured into one HIP graph (the operations only enqueue kernels) and the
    graph is replayed once untimed, then once timed between two device
    synchronizations.  Small workloads finish a step in less time than Python
    takes to issue one, so eager timing would measure the host."""
    import torch

    from paper_2512_22147_amd import mep

    call = S["call"]
    saved = call.stream
    s = torch.cuda.Stream()
    call.stream = s.cuda_stream
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for _ in range(steps):
            mep.mep_run(call)
    g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g.replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    call.stream = saved
    del g
    return elapsed * 1e3 / steps


def run_gpu(workload: str, dtype: str, steps: int, warmup: int, variant: int, eq3_flush: bool = True,
            graph: bool = False):
    import torch

    from paper_2512_22147_amd import mep

    S = setup(workload, dtype)
    code = S["code"]
    mep.mep_set_variant(code, variant)
    log(f"[bench] warmup {warmup} steps")
    for _ in range(warmup):
        S["step"]()
    torch.cuda.synchronize()
    # stamp every PROFILE_EVERY-th step (all of its streaming launches): an
    # event pair costs ~16 us of host time per launch, which would make small
    # workloads host-bound and adds ~1 us to a headline step
    nk = len(S["kernels"])
    stamped = (steps + PROFILE_EVERY - 1) // PROFILE_EVERY
    mep.mep_profile_begin_sampled(stamped * nk, nk, PROFILE_EVERY)
    log(f"[bench] timing {steps} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        S["step"]()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kern = S["kernels"]
    samples, kern_ms, launches = mep.mep_profile_end_samples(stamped * len(kern) + 16)
    config = mep.mep_variant_info(code, mep.dtype_code(S["tdt"]), S["m"], S["n"], max(variant, 0))
    ms_step = elapsed * 1e3 / steps
    ms_eager = ms_step
    if graph:
        ms_step = graph_step_ms(S, steps)
    eq3 = eq3_timing(S, ms_step) if eq3_flush else None
    mep.mep_set_variant(code, -1)
    per_kernel = []
    if launches == stamped * len(kern):
        # launch position p of every stamped step is the same kernel
        for p, (name, nbytes) in enumerate(kern):
            ms = sum(samples[p::len(kern)]) / stamped
            per_kernel.append({"kernel": name, "ms": ms, "alg_bytes": nbytes,
                               "gbs": nbytes / (ms * 1e-3) / 1e9})
        dom = max(per_kernel, key=lambda k: k["ms"])
    else:
        # a size whose path adds launches (e.g. a two-pass fallback): average them
        dom = {"kernel": kern[0][0], "ms": kern_ms / max(launches, 1), "alg_bytes": kern[0][1]}
        dom["gbs"] = dom["alg_bytes"] / (dom["ms"] * 1e-3) / 1e9
    res = {
        "dtype": dtype, "m": S["m"], "n": S["n"], "ms_per_step": ms_step, "ms_per_step_eager": ms_eager,
        "value_gbs": S["alg_step"] / (ms_step * 1e-3) / 1e9,
        "kernel_ms": dom["ms"], "kernel_launches": launches, "kernel_name": dom["kernel"],
        "kernel_gbs": dom["gbs"], "per_kernel": per_kernel if len(per_kernel) > 1 else None,
        "alg_bytes_step": S["alg_step"], "alg_bytes_kernel": dom["alg_bytes"], "config": config, "eq3": eq3,
        "outs": {k: v.cpu().numpy() for k, v in S["outs"]().items()},
        "host": S["host"], "w": S["w"],
    }
    del S
    torch.cuda.empty_cache()
    return res


def probe_copy():
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        mep.mep_stream_copy(src, dst)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    reps = 10
    for _ in range(reps):
        mep.mep_stream_copy(src, dst)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    log(f"[bench] copy probe: {nbytes} B read + {nbytes} B written per launch, "
        f"{2 * nbytes / dt / 1e9:.1f} GB/s")
    return {"bytes_read": nbytes, "bytes_written": nbytes, "gbs": 2 * nbytes / dt / 1e9}


def probe_floor(reps: int = 200):
    """The launch floor: `reps` launches of a 16-byte mep_stream_copy (one
    workgroup; one load and one store by the lane that has data) captured into
    one HIP graph and replayed, so that the host is out of the way; the time
    per launch is what any extra kernel of a step costs at least."""
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    src = torch.ones(16, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for _ in range(reps):
            mep.mep_stream_copy(src, dst, stream=s)
    g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g.replay()
    torch.cuda.synchronize()
    us = (time.perf_counter() - t0) * 1e6 / reps
    log(f"[bench] launch floor: {us:.2f} us per launch of a 16-byte copy (graph replay)")
    del g
    return {"kernel": "k_copy16 (16 bytes, one workgroup)", "launches": reps, "timing": "graph replay",
            "us_per_launch": round(us, 3)}


def mix_ceiling(read_gbs: float, copy_gbs: float, bytes_read: int, bytes_written: int):
    """Bandwidth bound of a kernel that reads R and writes W bytes, from the
    measured read ceiling and copy rate: the copy gives the time a written byte
    costs beside a read one (t_copy = N / read + N / write), and the kernel's
    bound is (R + W) / (R / read + W / write)."""
    t_read_byte = 1.0 / (read_gbs * 1e9)
    t_write_byte = 2.0 / (copy_gbs * 1e9) - t_read_byte
    if t_write_byte <= 0:
        return None
    t = bytes_read * t_read_byte + bytes_written * t_write_byte
    return {"read_gbs": read_gbs, "copy_gbs": copy_gbs, "write_gbs_derived": round(1.0 / t_write_byte / 1e9, 1),
            "bytes_read": bytes_read, "bytes_written": bytes_written,
            "mix_gbs": round((bytes_read + bytes_written) / t / 1e9, 1)}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def probe_read(n: int, dtype: str = "f32", reps: int = 20) -> float:
    """GB/s of the library's sum over n elements (a pure read of n * es
    bytes), launched back to back, so an array that fits the 256 MB Infinity
    Cache is read from there as a cache-resident matrix of the same size is."""
    import torch

    from paper_2512_22147_amd import mep

    dev = torch.device("cuda:0")
    tdt, code, es = (torch.float32, mep.MEP_F32, 4) if dtype == "f32" else (torch.float64, mep.MEP_F64, 8)
    x = torch.ones(n, dtype=tdt, device=dev)
    s = torch.empty(1, dtype=tdt, device=dev)
    ws = torch.empty(max(mep.mep_workspace_bytes(mep.MEP_OP_REDUCE_SUM, code, 1, n), 1),
                     dtype=torch.uint8, device=dev)
    call = mep.make_call(mep.MEP_OP_REDUCE_SUM, x, out0=s, ws=ws)
    for _ in range(3):
        mep.mep_run(call)
    torch.cuda.synchronize()
    mep.mep_profile_begin(reps)
    for _ in range(reps):
        mep.mep_run(call)
    torch.cuda.synchronize()
    tot, cnt = mep.mep_profile_end()
    del x, ws
    torch.cuda.empty_cache()
    return n * es / (tot / cnt * 1e-3) / 1e9


def stream_read_bytes(w, dtype: str) -> int:
    """Bytes the workload's dominant kernel streams from memory: the matrix
    (both for GESUMMV), the vector for the sum, both inputs for the add."""
    es = 4 if dtype == "f32" else 8
    if w.op == "reduce_sum":
        return w.n * es
    if w.op == "vector_add":
        return 2 * w.n * es
    return (2 if w.op == "axpby_mv" else 1) * w.m * w.n * es


def probe_ceiling(nbytes: int):
    """HBM read ceiling: the library's sum (a pure stream) over as many bytes
    as the workload's dominant kernel reads, so that the kernel is compared
    with a read of its own size (a 2 GiB stream reads a few % slower than a
    1 GiB one); at most the longest vector the library accepts, 65535 x 8192
    fp32 elements."""
    n = max(1, min(nbytes // 4, 65535 * 8192))
    gbs = probe_read(n)
    log(f"[bench] HBM ceiling probe: sum of {n * 4} B fp32, {gbs:.1f} GB/s")
    return {"kernel": f"k_reduce_sum (fp32, {n} elements)", "bytes_read": n * 4, "gbs": round(gbs, 1),
            "frac_of_peak": round(gbs / PEAK_GBS, 4)}


def cpu_baseline(res):
    import numpy as np

    import oracle

    w, host = res["w"], res["host"]
    host64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in host.items()}
    threads = oracle.default().num_threads()
    # Eq. 3 (R = 30, k = 3); each sample is `inner` back-to-back calls, sized
    # from the second of two untimed calls (the first also pays page faults)
    # so that the whole timed sample is 10-14 s of host time (R = 5, k = 1 when
    # one call alone is longer than 1 s)
    per = float("inf")
    for _ in range(2):
        t0 = time.perf_counter()
        ref = oracle_outputs(w, host64, res["dtype"])
        per = min(per, time.perf_counter() - t0)
    R, k = (30, 3) if per <= 1.0 else (5, 1)
    inner = max(1, int(math.ceil(14.0 / (R * max(per, 1e-6)))))
    log(f"[bench] CPU oracle ({cpu_model()}): {R} samples of {inner} calls on {threads} threads")
    times = []
    for _ in range(R):
        t0 = time.perf_counter()
        for _ in range(inner):
            ref = oracle_outputs(w, host64, res["dtype"])
        times.append((time.perf_counter() - t0) / inner)
    t = oracle.trimmed_mean(times, k)
    shape = "x".join(str(s) for s in next(iter(host.values())).shape)
    return {
        "value": res["alg_bytes_step"] / t / 1e9, "unit": "GB/s", "cores": threads,
        "kind": "oracle", "seconds_per_call": t, "cpu_model": cpu_model(),
        "sample": f"the full {w.name} workload ({shape} {res['dtype']}; inputs promoted to fp64 "
                  f"before timing): {R} samples of {inner} back-to-back calls ({R * inner} calls, "
                  f"~{R * inner * t:.0f} s) after two untimed calls, Eq. 3 trimmed mean with k={k}",
    }, ref


def fe_vs_oracle(res, ref):
    """Functional equivalence against the oracle (Eq. 4, normwise reading; the
    pass criterion) with two diagnostics beside it: the element-wise relative
    error max_i |out_i - ref_i| / |ref_i| and the condition-scaled error
    max_i |out_i - ref_i| / scale_i, where scale is the same operation on the
    absolute values of the inputs (|A|^T (|A| |x|) for ATAX); the worst output
    counts for each."""
    import numpy as np

    from paper_2512_22147_amd import mep

    tol = 1e-4 if res["dtype"] == "f32" else 1e-12
    absins = {k: np.abs(v) for k, v in res["host"].items()}
    scales = oracle_outputs(res["w"], absins, res["dtype"])
    worst = {"normwise": 0.0, "elementwise": 0.0, "condition_scaled": 0.0}
    for k, r in ref.items():
        out = np.asarray(res["outs"][k], np.float64).ravel()
        r = np.asarray(r, np.float64).ravel()
        d = np.abs(out - r)
        nz = r != 0
        sc = np.asarray(scales[k], np.float64).ravel()
        pos = sc > 0
        worst["normwise"] = max(worst["normwise"], mep.mep_check_fe(res["outs"][k], r, tol)[0])
        if nz.any():
            worst["elementwise"] = max(worst["elementwise"], float(np.max(d[nz] / np.abs(r[nz]))))
        cond = float(np.max(d[pos] / sc[pos])) if pos.any() else 0.0
        if (d[~pos] > 0).any():
            cond = float("inf")
        worst["condition_scaled"] = max(worst["condition_scaled"], cond)
    return {**{k: float(f"{v:.4g}") for k, v in worst.items()}, "tol": tol,
            "pass": worst["normwise"] <= tol}


# Eqs. 1-2 budget parameters; the paper gives no values, these are the
# defaults this harness reports against (flags only: the workload sizes are fixed)
T_MIN_MS = 0.010
T_MAX_S = 60.0
S_MAX_BYTES = 8 << 30


def mep_budget(w, dtype, kernel_ms, overall_s):
    """Eq. 1 (T_ker >= T_min, T_overall <= T_max) and Eq. 2 (S_data <= S_max)."""
    import numpy as np

    s_data = w.data_bytes(np.float32 if dtype == "f32" else np.float64)
    return {"T_ker_ms": round(kernel_ms, 5), "T_min_ms": T_MIN_MS, "T_ker_ok": kernel_ms >= T_MIN_MS,
            "T_overall_s": round(overall_s, 2), "T_max_s": T_MAX_S, "T_overall_ok": overall_s <= T_MAX_S,
            "S_data_bytes": s_data, "S_max_bytes": S_MAX_BYTES, "S_data_ok": s_data <= S_MAX_BYTES}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the row-sharded "
              "multi-GPU layout is a design, not a measured configuration", file=sys.stderr)
        sys.exit(2)
    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2512_22147_amd import datagen, mep

    mep.lib()
    if args.workload not in datagen.WORKLOADS:
        print(f"unknown workload {args.workload}; known: {sorted(datagen.WORKLOADS)}", file=sys.stderr)
        sys.exit(2)
    # the ceiling first: HBM throughput read right after minutes of streaming is a few % lower
    ceiling = None if args.no_ceiling else probe_ceiling(
        stream_read_bytes(datagen.WORKLOADS[args.workload], args.dtype))
    t_mep = time.perf_counter()
    prim = run_gpu(args.workload, args.dtype, args.steps, args.warmup, args.variant, not args.no_eq3)
    # the MEP proper: input generation, upload, warm-up and timed steps
    t_mep = time.perf_counter() - t_mep
    fe = None
    cpu = None
    if not args.no_cpu_baseline:
        cpu, ref = cpu_baseline(prim)
        fe = fe_vs_oracle(prim, ref)
    prim.pop("host")
    secondary = None
    if args.workload == HEADLINE and not args.no_f64 and args.dtype == "f32":
        sec = run_gpu(args.workload, "f64", args.steps, args.warmup, args.variant, not args.no_eq3)
        sec_fe = None
        if not args.no_cpu_baseline:
            import numpy as np

            host64 = {k: np.ascontiguousarray(v, dtype=np.float64) for k, v in sec["host"].items()}
            sec_fe = fe_vs_oracle(sec, oracle_outputs(sec["w"], host64, "f64"))
        sec.pop("host")
        secondary = {
            "dtype": "f64", "value": round(sec["value_gbs"], 1), "unit": "GB/s",
            "ms_per_step": round(sec["ms_per_step"], 4),
            "kernel_gbs": round(sec["kernel_gbs"], 1),
            "frac_of_peak": round(sec["kernel_gbs"] / PEAK_GBS, 4),
            "traffic": measured_traffic(args.workload, "f64", sec["config"]),
            "kernel_config": sec["config"], "eq3": sec["eq3"], "fe_vs_oracle": sec_fe,
        }
    others = None
    if args.workload == HEADLINE and not args.no_configs:
        others = []
        for wl, dt in OTHER_CONFIGS:
            r = run_gpu(wl, dt, args.steps, args.warmup, -1, False, graph=True)
            # a plain read of as many matrix bytes, from wherever they live
            # (HBM, or the Infinity Cache for matrices of at most 128 MiB)
            mats = 2 if r["w"].op == "axpby_mv" else 1
            read_gbs = probe_read(mats * r["m"] * r["n"], dt)
            others.append({
                "workload": wl, "dtype": dt, "m": r["m"], "n": r["n"],
                "ms_per_step": round(r["ms_per_step"], 5), "timing": "graph replay of the timed steps",
                "ms_per_step_eager": round(r["ms_per_step_eager"], 5),
                "value": round(r["value_gbs"], 1), "unit": "GB/s",
                "kernel_gbs": round(r["kernel_gbs"], 1), "kernel_frac": round(r["kernel_gbs"] / PEAK_GBS, 4),
                "kernel_config": r["config"], "same_size_read_gbs": round(read_gbs, 1),
                "kernel_frac_of_read": round(r["kernel_gbs"] / read_gbs, 4),
            })
    w0 = datagen.WORKLOADS[args.workload]
    # kernels that write as much as they read are bound by the read/write mix:
    # GEMVER's first pass (A read, Ahat written) and the vector add (2:1)
    mixed = w0.op in ("gemver", "vector_add")
    copy = probe_copy() if (args.probe_copy or mixed) else None
    floor = probe_floor() if args.probe_floor else None
    mix = None
    if mixed and ceiling is not None and copy is not None:
        es = 4 if args.dtype == "f32" else 8
        m_, n_ = prim["m"], prim["n"]
        if w0.op == "gemver":
            # pass 1: A, u1, u2, y read once, v1, v2 from L2; Ahat and the partials written
            rd, wr = (m_ * n_ + 3 * m_ + 2 * n_) * es, m_ * n_ * es
        else:
            rd, wr = 2 * n_ * es, n_ * es
        mix = mix_ceiling(ceiling["gbs"], copy["gbs"], rd, wr)
        if mix is not None:
            mix["kernel_frac_of_mix_ceiling"] = round(prim["kernel_gbs"] / mix["mix_gbs"], 4)
    selection = select_round(args.workload, args.dtype) if args.select else None
    w = prim["w"]
    desc = OPS[w.op][2]
    metric = (HEADLINE_METRIC if args.workload == HEADLINE and args.dtype == "f32"
              else f"achieved HBM GB/s (and % of MI355X peak) for {desc}, {args.dtype} {w.name}")
    out = {
        "metric": metric,
        "value": round(prim["value_gbs"], 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(prim["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic",
        "config": {"workload": f"{desc}, {w.name}: {w.note}; {w.dist} seed {w.seed}",
                   "m": prim["m"], "n": prim["n"], "seed": w.seed, "kernel_candidate": args.variant},
        "pct_of_peak": round(100.0 * prim["value_gbs"] / PEAK_GBS, 2),
        "roofline": {
            "bound": "hbm", "achieved": round(prim["kernel_gbs"], 1), "peak": PEAK_GBS, "unit": "GB/s",
            "frac": round(prim["kernel_gbs"] / PEAK_GBS, 4),
            "traffic": measured_traffic(args.workload, args.dtype, prim["config"]),
            "kernel": prim["kernel_name"], "kernel_config": prim["config"],
            "kernel_ms": round(prim["kernel_ms"], 5),
            "alg_bytes_per_launch": prim["alg_bytes_kernel"],
        },
        "per_kernel": None if prim["per_kernel"] is None else [
            {"kernel": k["kernel"], "ms": round(k["ms"], 5), "alg_bytes": k["alg_bytes"],
             "gbs": round(k["gbs"], 1), "frac": round(k["gbs"] / PEAK_GBS, 4)} for k in prim["per_kernel"]],
        "eq3": prim["eq3"],
        "selection": selection,
        "cpu_baseline": cpu,
        "fe_error_vs_oracle": None if fe is None else fe["normwise"],
        "fe_vs_oracle": fe,
        "secondary": secondary,
        "other_configs": others,
        "copy_probe": copy,
        "launch_floor": floor,
        "mix_ceiling": mix,
        "hbm_ceiling_probe": ceiling,
        "mep_budget": mep_budget(w, args.dtype, prim["kernel_ms"], t_mep),
        "kernel_frac_of_ceiling": None if ceiling is None else round(prim["kernel_gbs"] / ceiling["gbs"], 4),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
