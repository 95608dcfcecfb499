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
    """Runs op on the GPU and returns host numpy outputs.  Inputs may be host
    arrays (copied to the GPU) or tensors already there (used as they are:
    no operation writes its inputs)."""
    import torch

    from paper_2512_22147_amd import mep

    dev = dev or torch.device("cuda:0")
    T = {k: v if torch.is_tensor(v) else torch.from_numpy(np.ascontiguousarray(v)).to(dev)
         for k, v in ins.items()}
    m, n = T["A"].shape
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


def condition_scales(op, ins, dt, alpha=ALPHA, beta=BETA):
    """Per-element error scales of each output: the same operation on the
    absolute values of every input (and |alpha|, |beta|), in the oracle --
    |A| |x| for y = A x, |A|^T (|A| |x|) for ATAX, |alpha| |A| |x| + |beta|
    |B| |x| for GESUMMV, and so on.  Any summation order of depth d keeps
    |out_i - exact_i| <= gamma_d * scale_i (first order)."""
    absins = {k: np.abs(v) for k, v in ins.items()}
    return oracle_outputs(op, absins, dt, alpha=abs(alpha), beta=abs(beta))


def diagnostics(got, ref, scale=None):
    """(normwise, element-wise relative, condition-scaled) error of one output.
    Element-wise: max |out_i - ref_i| / |ref_i| over ref_i != 0 (fails even for
    correct fp32 results near zero, so it is logged only).  Condition-scaled:
    max |out_i - ref_i| / scale_i (+inf where scale_i = 0 and out_i != ref_i)."""
    out = np.asarray(got, np.float64).ravel()
    r = np.asarray(ref, np.float64).ravel()
    d = np.abs(out - r)
    nz = r != 0
    elem = float(np.max(d[nz] / np.abs(r[nz]))) if nz.any() else 0.0
    cond = None
    if scale is not None:
        sc = np.asarray(scale, np.float64).ravel()
        pos = sc > 0
        cond = float(np.max(d[pos] / sc[pos])) if pos.any() else 0.0
        if (d[~pos] > 0).any():
            cond = float("inf")
    return normwise(out, r), elem, cond


def cond_bound(m, n, dt):
    """A rigorous bound on the condition-scaled error of any of these
    operations: no output passes through more than m + n + 64 roundings
    (a row dot of n terms, a column sum of m, the partial-sum stages and
    epilogues); twice gamma_d, since the fp64 oracle's own error is of the
    same order as an fp64 GPU result's."""
    u = {np.dtype(np.float32): 2.0**-24, np.dtype(np.float64): 2.0**-53}[np.dtype(dt)]
    d = m + n + 64
    return 2.0 * d * u / (1.0 - d * u)


def assert_parity(op, got, ref, dt, what="", scales=None, dims=None):
    """Normwise error <= TOL is the pass criterion; the element-wise and
    condition-scaled errors are printed beside it, and with `scales` (from
    condition_scales) and `dims` = (m, n) the condition-scaled error must also
    stay within cond_bound -- a per-element check that bites on outputs whose
    own scale is far below max|ref| (with inputs of one magnitude it is the
    looser of the two)."""
    tol = TOL[dt]
    for k, r in ref.items():
        assert got[k].shape == r.shape, f"{what} {k}: shape {got[k].shape} vs {r.shape}"
        err, elem, cond = diagnostics(got[k], r, None if scales is None else scales[k])
        print(f"parity {what} {op} {k}: normwise {err:.3e} elementwise {elem:.3e} "
              f"condition-scaled {'-' if cond is None else f'{cond:.3e}'}")
        assert err <= tol, (f"{what} {op} {k}: normwise error {err:.3e} > {tol:.0e} "
                            f"(elementwise {elem:.3e}, condition-scaled {cond})")
        if cond is not None and dims is not None:
            bound = cond_bound(dims[0], dims[1], dt)
            assert cond <= bound, f"{what} {op} {k}: condition-scaled error {cond:.3e} > {bound:.3e}"
