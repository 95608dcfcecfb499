"""Shared helpers of the GPU parity tests: run an operation through the
C-ABI (via the binding) and through the CPU oracle on the same inputs."""
from __future__ import annotations

import numpy as np

import oracle

TOL = {np.float32: 1e-4, np.float64: 1e-12}
OPS = ("matvec", "matvec_t", "bicg", "ata_x", "axpby_mv", "gemver")


def op_code(op):
    from paper_2512_22147_amd import mep

    return {"matvec": mep.MEP_OP_MATVEC, "matvec_t": mep.MEP_OP_MATVEC_T, "bicg": mep.MEP_OP_BICG,
            "ata_x": mep.MEP_OP_ATA_X, "axpby_mv": mep.MEP_OP_AXPBY_MV,
            "gemver": mep.MEP_OP_GEMVER}[op]


def make_inputs(op, m, n, dt, seed, kind="uniform"):
    from paper_2512_22147_amd import datagen

    draw = {"uniform": datagen.uniform, "normal": datagen.normal, "ternary": datagen.ternary}[kind]
    ins = {"A": draw(seed, 0, (m, n), dt)}
    if op in ("matvec", "ata_x", "axpby_mv", "bicg"):
        ins["x"] = draw(seed, 1, (n,), dt)
    if op in ("matvec_t", "bicg"):
        ins["w"] = draw(seed, 2, (m,), dt)
    if op == "axpby_mv":
        ins["B"] = draw(seed, 3, (m, n), dt)
    if op == "gemver":
        for aid, (name, ln) in enumerate((("u1", m), ("v1", n), ("u2", m), ("v2", n), ("y", m),
                                          ("z", n)), start=4):
            ins[name] = draw(seed, aid, (ln,), dt)
    return ins


ALPHA, BETA = 1.5, 1.2


def oracle_outputs(op, ins, dt, alpha=ALPHA, beta=BETA):
    A = ins["A"]
    if op == "matvec":
        return {"y": oracle.matvec(A, ins["x"])}
    if op == "matvec_t":
        return {"z": oracle.matvec_t(A, ins["w"])}
    if op == "bicg":
        q, s = oracle.bicg(A, ins["x"], ins["w"])
        return {"z": s, "q": q}
    if op == "ata_x":
        y, t = oracle.ata_x(A, ins["x"])
        return {"y": y, "t": t}
    if op == "axpby_mv":
        a = oracle.elem_scalar(alpha, dt)
        b = oracle.elem_scalar(beta, dt)
        return {"y": oracle.axpby_mv(a, A, b, ins["B"], ins["x"])}
    if op == "gemver":
        a = oracle.elem_scalar(alpha, dt)
        b = oracle.elem_scalar(beta, dt)
        Ahat, x, w = oracle.gemver(a, b, A, ins["u1"], ins["v1"], ins["u2"], ins["v2"], ins["y"],
                                   ins["z"])
        return {"Ahat": Ahat, "x": x, "w": w}
    raise ValueError(op)


def gpu_outputs(op, ins, dt, alpha=ALPHA, beta=BETA, dev=None):
    """Runs op on the GPU and returns host numpy outputs."""
    import torch

    from paper_2512_22147_amd import mep

    dev = dev or torch.device("cuda:0")
    T = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in ins.items()}
    m, n = ins["A"].shape
    if op == "matvec":
        out = {"y": mep.mep_matvec(T["A"], T["x"])}
    elif op == "matvec_t":
        out = {"z": mep.mep_matvec_t(T["A"], T["w"])}
    elif op == "bicg":
        z, q = mep.mep_matvec_t(T["A"], T["w"], p=T["x"])
        out = {"z": z, "q": q}
    elif op == "ata_x":
        t = torch.empty(m, dtype=T["A"].dtype, device=dev)
        y = mep.mep_ata_x(T["A"], T["x"], t=t)
        out = {"y": y, "t": t}
    elif op == "axpby_mv":
        out = {"y": mep.mep_axpby_mv(alpha, T["A"], beta, T["B"], T["x"])}
    elif op == "gemver":
        Ahat, x, w = mep.mep_gemver(alpha, beta, T["A"], T["u1"], T["v1"], T["u2"], T["v2"], T["y"],
                                    T["z"])
        out = {"Ahat": Ahat, "x": x, "w": w}
    else:
        raise ValueError(op)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def normwise(out, ref):
    out = np.asarray(out, np.float64)
    ref = np.asarray(ref, np.float64)
    if out.size == 0:
        return 0.0
    if not np.isfinite(out).all():
        return float("inf")
    scale = float(np.max(np.abs(ref)))
    worst = float(np.max(np.abs(out - ref)))
    if scale == 0.0:
        return 0.0 if worst == 0.0 else float("inf")
    return worst / scale


def assert_parity(op, got, ref, dt, what=""):
    tol = TOL[dt]
    for k, r in ref.items():
        assert got[k].shape == r.shape, f"{what} {k}: shape {got[k].shape} vs {r.shape}"
        err = normwise(got[k], r)
        assert err <= tol, f"{what} {op} {k}: normwise error {err:.3e} > {tol:.0e}"
