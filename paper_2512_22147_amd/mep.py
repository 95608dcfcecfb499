"""Python binding of libmep.so (include/mep.h): argument marshalling only.

Every computation runs in the library's HIP kernels; PyTorch only provides
device memory and the stream.  The functions keep the C names.  Loading
fails loudly when ``libmep.so`` has not been built: there is no fallback.

Tensors passed to the operations must be contiguous CUDA (HIP) tensors of
dtype float32 or float64.  Outputs and the workspace are allocated with torch
when not given.  Operations are asynchronous on ``stream`` (default: torch's
current stream), like the C functions.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmep.so")

MEP_F32, MEP_F64 = 0, 1
MEP_OK, MEP_EINVAL, MEP_EALIGN, MEP_EWORKSPACE, MEP_EHIP, MEP_EBUDGET = range(6)
(MEP_OP_MATVEC, MEP_OP_MATVEC_T, MEP_OP_BICG, MEP_OP_ATA_X, MEP_OP_AXPBY_MV, MEP_OP_REDUCE_SUM,
 MEP_OP_VECTOR_ADD, MEP_OP_GEMVER) = range(8)
ERROR_NAMES = {1: "MEP_EINVAL", 2: "MEP_EALIGN", 3: "MEP_EWORKSPACE", 4: "MEP_EHIP", 5: "MEP_EBUDGET"}

# Names exported by libmep.so, in the order include/mep.h declares them.
EXPORTS = (
    "mep_workspace_bytes", "mep_matvec", "mep_matvec_t", "mep_ata_x", "mep_axpby_mv",
    "mep_run", "mep_time_trimmed", "mep_trimmed_mean", "mep_check_fe",
    "mep_variant_count", "mep_set_variant", "mep_variant_info", "mep_profile_begin", "mep_profile_end",
    "mep_stream_copy", "mep_last_error", "mep_version", "mep_select_variant",
    "mep_reduce_sum", "mep_vector_add", "mep_gemver", "mep_profile_end_samples", "mep_profile_begin_sampled",
    "mep_ata_x_noalloc",
)
NOALLOC_SCRATCH_BYTES = 64 << 20  # MEP_NOALLOC_SCRATCH_BYTES


class MepError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {message}")
        self.code = code


class MepCall(ctypes.Structure):
    """mep_call_t."""
    _fields_ = [
        ("op", ctypes.c_int), ("dtype", ctypes.c_int),
        ("m", ctypes.c_int64), ("n", ctypes.c_int64),
        ("A", ctypes.c_void_p), ("B", ctypes.c_void_p),
        ("in0", ctypes.c_void_p), ("in1", ctypes.c_void_p),
        ("out0", ctypes.c_void_p), ("out1", ctypes.c_void_p),
        ("alpha", ctypes.c_double), ("beta", ctypes.c_double),
        ("ws", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t),
        ("stream", ctypes.c_void_p),
        ("flush_buf", ctypes.c_void_p), ("flush_bytes", ctypes.c_size_t),
        ("in2", ctypes.c_void_p), ("in3", ctypes.c_void_p), ("in4", ctypes.c_void_p),
        ("in5", ctypes.c_void_p), ("out2", ctypes.c_void_p),
    ]


class MepCandidateResult(ctypes.Structure):
    """mep_candidate_result_t."""
    _fields_ = [("mean_ms", ctypes.c_double), ("fe_err", ctypes.c_double), ("fe_pass", ctypes.c_int)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library with typed entry points."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2512_22147_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    i, i64, vp, d, sz = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_double, ctypes.c_size_t
    L.mep_workspace_bytes.argtypes = [i, i, i64, i64]
    L.mep_workspace_bytes.restype = sz
    L.mep_matvec.argtypes = [i, i64, i64, vp, vp, vp, vp, sz, vp]
    L.mep_matvec_t.argtypes = [i, i64, i64, vp, vp, vp, vp, vp, vp, sz, vp]
    L.mep_ata_x.argtypes = [i, i64, i64, vp, vp, vp, vp, vp, sz, vp]
    L.mep_axpby_mv.argtypes = [i, i64, i64, d, vp, d, vp, vp, vp, vp, sz, vp]
    L.mep_ata_x_noalloc.argtypes = [i, i64, i64, vp, vp, vp, vp, vp]
    L.mep_run.argtypes = [ctypes.POINTER(MepCall)]
    L.mep_time_trimmed.argtypes = [ctypes.POINTER(MepCall), i, i, i, i, i,
                                   ctypes.POINTER(d), ctypes.POINTER(d)]
    L.mep_trimmed_mean.argtypes = [ctypes.POINTER(d), i, i]
    L.mep_trimmed_mean.restype = d
    L.mep_check_fe.argtypes = [i, vp, ctypes.POINTER(d), i64, d, ctypes.POINTER(d),
                               ctypes.POINTER(ctypes.c_int)]
    L.mep_variant_count.argtypes = [i, i, i64, i64]
    L.mep_set_variant.argtypes = [i, i]
    L.mep_variant_info.argtypes = [i, i, i64, i64, i, ctypes.c_char_p, sz]
    L.mep_profile_begin.argtypes = [i]
    L.mep_profile_begin_sampled.argtypes = [i, i, i]
    L.mep_profile_end.argtypes = [ctypes.POINTER(d), ctypes.POINTER(ctypes.c_int)]
    L.mep_stream_copy.argtypes = [vp, vp, sz, vp]
    L.mep_reduce_sum.argtypes = [i, i64, vp, vp, vp, sz, vp]
    L.mep_vector_add.argtypes = [i, i64, vp, vp, vp, vp]
    L.mep_gemver.argtypes = [i, i64, i64, d, d, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.mep_profile_end_samples.argtypes = [ctypes.POINTER(d), i, ctypes.POINTER(d),
                                          ctypes.POINTER(ctypes.c_int)]
    L.mep_select_variant.argtypes = [ctypes.POINTER(MepCall), i, i, i, i, i, d, i,
                                     ctypes.POINTER(ctypes.c_int), ctypes.POINTER(MepCandidateResult), i]
    L.mep_last_error.restype = ctypes.c_char_p
    L.mep_version.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(rc: int) -> None:
    if rc != MEP_OK:
        raise MepError(rc, lib().mep_last_error().decode())


def mep_last_error() -> str:
    return lib().mep_last_error().decode()


def mep_version() -> str:
    return lib().mep_version().decode()


# ---------------------------------------------------------------------------
# torch marshalling
# ---------------------------------------------------------------------------

def _torch():
    import torch

    return torch


def dtype_code(dtype) -> int:
    torch = _torch()
    if dtype == torch.float32:
        return MEP_F32
    if dtype == torch.float64:
        return MEP_F64
    raise TypeError(f"unsupported dtype {dtype}; use float32 or float64")


def _ptr(t) -> int:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr() if t.numel() > 0 else None


def _matrix(A, name="A"):
    """(m, n) of a 2-D float32/float64 matrix."""
    if A is None or A.dim() != 2:
        raise ValueError(f"{name} must be a 2-D tensor")
    dtype_code(A.dtype)
    return int(A.shape[0]), int(A.shape[1])


def _like(t, name, length, ref):
    """Checks that t has `length` elements and ref's dtype and device, before
    any pointer reaches the C ABI (which only sees addresses and sizes: a
    short or mistyped buffer would be read or written past its end)."""
    if t is None:
        return
    if t.dtype != ref.dtype:
        raise ValueError(f"{name} is {t.dtype}, expected {ref.dtype}")
    if t.numel() != length:
        raise ValueError(f"{name} has {t.numel()} elements, expected {length}")
    if t.device != ref.device:
        raise ValueError(f"{name} is on {t.device}, expected {ref.device}")


def _same_shape(t, name, ref):
    if t is None:
        return
    if tuple(t.shape) != tuple(ref.shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(ref.shape)}")
    _like(t, name, ref.numel(), ref)


def _ws_checked(ws, ref):
    if ws is not None and ws.device != ref.device:
        raise ValueError(f"ws is on {ws.device}, expected {ref.device}")


def _stream(stream) -> int:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _ws(op, A, ws):
    torch = _torch()
    m, n = A.shape
    _ws_checked(ws, A)
    need = mep_workspace_bytes(op, dtype_code(A.dtype), m, n)
    if ws is None and need > 0:
        ws = torch.empty(need, dtype=torch.uint8, device=A.device)
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    return ws, nbytes


def _out(like, n, out):
    torch = _torch()
    if out is None:
        out = torch.empty(n, dtype=like.dtype, device=like.device)
    return out


def mep_workspace_bytes(op: int, dtype: int, m: int, n: int) -> int:
    return int(lib().mep_workspace_bytes(op, dtype, m, n))


def mep_matvec(A, x, y=None, ws=None, stream=None):
    """y = A x."""
    m, n = _matrix(A)
    _like(x, "x", n, A)
    _like(y, "y", m, A)
    y = _out(A, m, y)
    ws, wsb = _ws(MEP_OP_MATVEC, A, ws)
    _check(lib().mep_matvec(dtype_code(A.dtype), m, n, _ptr(A), _ptr(x), _ptr(y),
                            _ptr(ws), wsb, _stream(stream)))
    return y


def mep_matvec_t(A, w, z=None, p=None, q=None, ws=None, stream=None):
    """z = A^T w; with p, also q = A p in the same read of A (BICG)."""
    m, n = _matrix(A)
    _like(w, "w", m, A)
    _like(z, "z", n, A)
    _like(p, "p", n, A)
    _like(q, "q", m, A)
    if q is not None and p is None:
        raise ValueError("q is only written with p (the paired product)")
    z = _out(A, n, z)
    if p is not None and q is None:
        q = _out(A, m, None)
    ws, wsb = _ws(MEP_OP_BICG if p is not None else MEP_OP_MATVEC_T, A, ws)
    _check(lib().mep_matvec_t(dtype_code(A.dtype), m, n, _ptr(A), _ptr(w), _ptr(z),
                              _ptr(p), _ptr(q), _ptr(ws), wsb, _stream(stream)))
    return (z, q) if p is not None else z


def mep_ata_x(A, x, y=None, t=None, ws=None, stream=None):
    """y = A^T (A x); t (optional) receives A x."""
    m, n = _matrix(A)
    _like(x, "x", n, A)
    _like(y, "y", n, A)
    _like(t, "t", m, A)
    y = _out(A, n, y)
    ws, wsb = _ws(MEP_OP_ATA_X, A, ws)
    _check(lib().mep_ata_x(dtype_code(A.dtype), m, n, _ptr(A), _ptr(x), _ptr(y), _ptr(t),
                           _ptr(ws), wsb, _stream(stream)))
    return y


def mep_ata_x_noalloc(A, x, y, t=None, stream=None):
    """y = A^T (A x) through the allocation-free entry point: the caller
    passes every output (y, and t if wanted); the library's own per-GPU
    scratch replaces the workspace.  Calls that overlap on one GPU race."""
    m, n = _matrix(A)
    _like(x, "x", n, A)
    if y is None:
        raise ValueError("y must be given: this entry point allocates nothing")
    _like(y, "y", n, A)
    _like(t, "t", m, A)
    _check(lib().mep_ata_x_noalloc(dtype_code(A.dtype), m, n, _ptr(A), _ptr(x), _ptr(y), _ptr(t),
                                   _stream(stream)))
    return y


def mep_axpby_mv(alpha, A, beta, B, x, y=None, ws=None, stream=None):
    """y = alpha A x + beta B x."""
    m, n = _matrix(A)
    _same_shape(B, "B", A)
    _like(x, "x", n, A)
    _like(y, "y", m, A)
    y = _out(A, m, y)
    ws, wsb = _ws(MEP_OP_AXPBY_MV, A, ws)
    _check(lib().mep_axpby_mv(dtype_code(A.dtype), m, n, float(alpha), _ptr(A), float(beta),
                              _ptr(B), _ptr(x), _ptr(y), _ptr(ws), wsb, _stream(stream)))
    return y


def mep_gemver(alpha, beta, A, u1, v1, u2, v2, y, z, x=None, w=None, Ahat=None, ws=None, stream=None):
    """GEMVER: Ahat = A + u1 v1^T + u2 v2^T, x = beta Ahat^T y + z, w = alpha Ahat x.

    Returns (Ahat, x, w).  Pass ``Ahat=A`` for the in-place update."""
    torch = _torch()
    m, n = _matrix(A)
    for name, v, ln in (("u1", u1, m), ("v1", v1, n), ("u2", u2, m), ("v2", v2, n), ("y", y, m),
                        ("z", z, n), ("x", x, n), ("w", w, m)):
        _like(v, name, ln, A)
    _same_shape(Ahat, "Ahat", A)
    if Ahat is None:
        Ahat = torch.empty_like(A)
    x = _out(A, n, x)
    w = _out(A, m, w)
    ws, wsb = _ws(MEP_OP_GEMVER, A, ws)
    _check(lib().mep_gemver(dtype_code(A.dtype), m, n, float(alpha), float(beta), _ptr(A), _ptr(Ahat),
                            _ptr(u1), _ptr(v1), _ptr(u2), _ptr(v2), _ptr(y), _ptr(z), _ptr(x), _ptr(w),
                            _ptr(ws), wsb, _stream(stream)))
    return Ahat, x, w


def mep_reduce_sum(x, s=None, ws=None, stream=None):
    """s = sum of x (one-element tensor)."""
    torch = _torch()
    dtype_code(x.dtype)
    n = x.numel()
    _like(s, "s", 1, x)
    _ws_checked(ws, x)
    if s is None:
        s = torch.empty(1, dtype=x.dtype, device=x.device)
    need = mep_workspace_bytes(MEP_OP_REDUCE_SUM, dtype_code(x.dtype), 1, n)
    if ws is None and need > 0:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().mep_reduce_sum(dtype_code(x.dtype), n, _ptr(x), _ptr(s), _ptr(ws), wsb,
                                _stream(stream)))
    return s


def mep_vector_add(a, b, c=None, stream=None):
    """c = a + b."""
    torch = _torch()
    dtype_code(a.dtype)
    _like(b, "b", a.numel(), a)
    _like(c, "c", a.numel(), a)
    if c is None:
        c = torch.empty_like(a)
    _check(lib().mep_vector_add(dtype_code(a.dtype), a.numel(), _ptr(a), _ptr(b), _ptr(c),
                                _stream(stream)))
    return c


def make_call(op, A, in0=None, in1=None, out0=None, out1=None, B=None, alpha=0.0, beta=0.0,
              ws=None, stream=None, flush_buf=None, in2=None, in3=None, in4=None, in5=None,
              out2=None) -> MepCall:
    """A mep_call_t over torch tensors (kept alive by the caller).

    GEMVER: in0..in5 = u1, v1, u2, v2, y, z; out0 = x, out1 = w, out2 = Ahat."""
    if op in (MEP_OP_REDUCE_SUM, MEP_OP_VECTOR_ADD):
        # vector samples: A is the first input vector; m = 1, n = its length
        torch = _torch()
        m, n = 1, A.numel()
        in0 = A if in0 is None else in0
        A = None
        dtype_code(in0.dtype)
        _like(in0, "in0", n, in0)
        if op == MEP_OP_REDUCE_SUM:
            _like(out0, "out0", 1, in0)
        else:
            _like(in1, "in1", n, in0)
            _like(out0, "out0", n, in0)
        _ws_checked(ws, in0)
        need = mep_workspace_bytes(op, dtype_code(in0.dtype), m, n)
        if ws is None and need > 0:
            ws = torch.empty(need, dtype=torch.uint8, device=in0.device)
        wsb = 0 if ws is None else ws.numel() * ws.element_size()
        dt = dtype_code(in0.dtype)
    else:
        m, n = _matrix(A)
        # expected lengths of in0.., out0.. per op (None: not used by the op)
        lengths = {
            MEP_OP_MATVEC: ({"in0": n}, {"out0": m}),
            MEP_OP_MATVEC_T: ({"in0": m}, {"out0": n}),
            MEP_OP_BICG: ({"in0": m, "in1": n}, {"out0": n, "out1": m}),
            MEP_OP_ATA_X: ({"in0": n}, {"out0": n, "out1": m}),
            MEP_OP_AXPBY_MV: ({"in0": n}, {"out0": m}),
            MEP_OP_GEMVER: ({"in0": m, "in1": n, "in2": m, "in3": n, "in4": m, "in5": n},
                            {"out0": n, "out1": m, "out2": m * n}),
        }
        if op not in lengths:
            raise ValueError(f"unknown op {op}")
        given = {"in0": in0, "in1": in1, "in2": in2, "in3": in3, "in4": in4, "in5": in5,
                 "out0": out0, "out1": out1, "out2": out2}
        ins, outs = lengths[op]
        for name, t in given.items():
            want = ins.get(name, outs.get(name))
            if want is None:
                if t is not None:
                    raise ValueError(f"{name} is not used by op {op}")
            else:
                _like(t, name, want, A)
        if op == MEP_OP_AXPBY_MV:
            _same_shape(B, "B", A)
        elif B is not None:
            raise ValueError(f"B is not used by op {op}")
        ws, wsb = _ws(op, A, ws)
        dt = dtype_code(A.dtype)
    c = MepCall()
    c.op, c.dtype, c.m, c.n = op, dt, m, n
    c.A, c.B = _ptr(A), _ptr(B)
    c.in0, c.in1, c.out0, c.out1 = _ptr(in0), _ptr(in1), _ptr(out0), _ptr(out1)
    c.in2, c.in3, c.in4, c.in5, c.out2 = _ptr(in2), _ptr(in3), _ptr(in4), _ptr(in5), _ptr(out2)
    c.alpha, c.beta = float(alpha), float(beta)
    c.ws, c.ws_bytes = _ptr(ws), wsb
    c.stream = _stream(stream)
    if flush_buf is not None:
        c.flush_buf = _ptr(flush_buf)
        c.flush_bytes = flush_buf.numel() * flush_buf.element_size()
    c._keep = ws  # the workspace must outlive the call
    return c


def mep_run(call: MepCall) -> None:
    _check(lib().mep_run(ctypes.byref(call)))


def mep_time_trimmed(call: MepCall, warmup: int = 3, R: int = 30, k: int = 3, inner: int = 1,
                     flush: bool = False):
    """Eq. 3 timing: returns (trimmed mean ms, list of R sample ms)."""
    mean = ctypes.c_double()
    samples = (ctypes.c_double * max(R, 1))()
    _check(lib().mep_time_trimmed(ctypes.byref(call), warmup, R, k, inner, int(bool(flush)),
                                  ctypes.byref(mean), samples))
    return mean.value, list(samples[:R])


def mep_trimmed_mean(samples, k: int) -> float:
    arr = (ctypes.c_double * max(len(samples), 1))(*[float(v) for v in samples])
    return float(lib().mep_trimmed_mean(arr, len(samples), k))


def mep_check_fe(out, ref, tol: float, dtype: Optional[int] = None):
    """Eq. 4 check of a host output against a host fp64 reference.

    ``out`` is a numpy array (float32/float64) or a torch tensor (copied to
    the host); returns (error, passed)."""
    import numpy as np

    if hasattr(out, "detach"):
        out = out.detach().cpu().numpy()
    out = np.ascontiguousarray(out)
    if dtype is None:
        dtype = MEP_F32 if out.dtype == np.float32 else MEP_F64
    ref = np.ascontiguousarray(ref, dtype=np.float64)
    if out.size != ref.size:
        raise ValueError("out and ref differ in length")
    err = ctypes.c_double()
    ok = ctypes.c_int()
    _check(lib().mep_check_fe(dtype, out.ctypes.data if out.size else None,
                              ref.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if ref.size else None,
                              out.size, float(tol), ctypes.byref(err), ctypes.byref(ok)))
    return err.value, bool(ok.value)


def mep_select_variant(call: MepCall, warmup: int = 3, R: int = 30, k: int = 3, inner: int = 1,
                       flush: bool = False, tol: float = 1e-4, apply: bool = False):
    """Eqs. 3-5 over the library's candidate kernels; returns (best, per-candidate
    list of (trimmed mean ms, FE error, FE passed))."""
    count = mep_variant_count(call.op, call.dtype, call.m, call.n)
    res = (MepCandidateResult * max(count, 1))()
    best = ctypes.c_int(-1)
    _check(lib().mep_select_variant(ctypes.byref(call), warmup, R, k, inner, int(bool(flush)),
                                    float(tol), int(bool(apply)), ctypes.byref(best), res, count))
    return best.value, [(r.mean_ms, r.fe_err, bool(r.fe_pass)) for r in res[:count]]


def mep_variant_count(op: int, dtype: int, m: int, n: int) -> int:
    return int(lib().mep_variant_count(op, dtype, m, n))


def mep_variant_info(op: int, dtype: int, m: int, n: int, variant: int) -> str:
    buf = ctypes.create_string_buffer(256)
    _check(lib().mep_variant_info(op, dtype, m, n, variant, buf, 256))
    return buf.value.decode()


def mep_set_variant(op: int, variant: int) -> None:
    _check(lib().mep_set_variant(op, variant))


def mep_profile_begin(capacity: int) -> None:
    _check(lib().mep_profile_begin(capacity))


def mep_profile_begin_sampled(capacity: int, group: int, every: int) -> None:
    """Stamp launch i (counted from here) when (i // group) % every == 0."""
    _check(lib().mep_profile_begin_sampled(capacity, group, every))


def mep_profile_end():
    """Returns (summed streaming-kernel ms, number of launches)."""
    tot = ctypes.c_double()
    cnt = ctypes.c_int()
    _check(lib().mep_profile_end(ctypes.byref(tot), ctypes.byref(cnt)))
    return tot.value, cnt.value


def mep_profile_end_samples(cap: int = 4096):
    """Returns (list of per-launch ms in launch order, summed ms, launches)."""
    tot = ctypes.c_double()
    cnt = ctypes.c_int()
    buf = (ctypes.c_double * max(cap, 1))()
    _check(lib().mep_profile_end_samples(buf, cap, ctypes.byref(tot), ctypes.byref(cnt)))
    return list(buf[:min(cap, cnt.value)]), tot.value, cnt.value


def mep_stream_copy(src, dst, stream=None) -> None:
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst smaller than src")
    if dst.device != src.device:
        raise ValueError(f"dst is on {dst.device}, expected {src.device}")
    _check(lib().mep_stream_copy(_ptr(src), _ptr(dst), nbytes, _stream(stream)))
