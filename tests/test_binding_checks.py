"""The Python binding checks every tensor's length, dtype and device before a
pointer reaches the C ABI (which sees only addresses and sizes).  Runs on the
CPU: each bad call must raise ValueError before anything touches a GPU, and
a call whose tensors are all well formed but live on the host must still be
refused (no host path exists)."""
import pytest
import torch

from paper_2512_22147_amd import mep

m, n = 6, 8


def f32(*shape):
    return torch.zeros(*shape, dtype=torch.float32)


def f64(*shape):
    return torch.zeros(*shape, dtype=torch.float64)


BAD_CALLS = {
    "matvec short x": lambda: mep.mep_matvec(f32(m, n), f32(n - 1)),
    "matvec long y": lambda: mep.mep_matvec(f32(m, n), f32(n), y=f32(m + 1)),
    "matvec fp64 x": lambda: mep.mep_matvec(f32(m, n), f64(n)),
    "matvec 1-D A": lambda: mep.mep_matvec(f32(m * n), f32(n)),
    "matvec_t short w": lambda: mep.mep_matvec_t(f32(m, n), f32(m - 1)),
    "matvec_t z of m": lambda: mep.mep_matvec_t(f32(m, n), f32(m), z=f32(m)),
    "bicg p of m": lambda: mep.mep_matvec_t(f32(m, n), f32(m), p=f32(m)),
    "bicg q of n": lambda: mep.mep_matvec_t(f32(m, n), f32(m), p=f32(n), q=f32(n)),
    "bicg q without p": lambda: mep.mep_matvec_t(f32(m, n), f32(m), q=f32(m)),
    "ata_x x of m": lambda: mep.mep_ata_x(f32(m, n), f32(m)),
    "ata_x t of n": lambda: mep.mep_ata_x(f32(m, n), f32(n), t=f32(n)),
    "ata_x fp64 y": lambda: mep.mep_ata_x(f32(m, n), f32(n), y=f64(n)),
    "axpby B transposed": lambda: mep.mep_axpby_mv(1.0, f32(m, n), 1.0, f32(n, m), f32(n)),
    "axpby B fp64": lambda: mep.mep_axpby_mv(1.0, f32(m, n), 1.0, f64(m, n), f32(n)),
    "gemver v1 of m": lambda: mep.mep_gemver(1.0, 1.0, f32(m, n), f32(m), f32(m), f32(m), f32(n),
                                             f32(m), f32(n)),
    "gemver Ahat shape": lambda: mep.mep_gemver(1.0, 1.0, f32(m, n), f32(m), f32(n), f32(m), f32(n),
                                                f32(m), f32(n), Ahat=f32(n, m)),
    "reduce s of 2": lambda: mep.mep_reduce_sum(f32(n), s=f32(2)),
    "vector_add short b": lambda: mep.mep_vector_add(f32(n), f32(n - 1)),
    "vector_add fp64 c": lambda: mep.mep_vector_add(f32(n), f32(n), c=f64(n)),
    "call matvec short x": lambda: mep.make_call(mep.MEP_OP_MATVEC, f32(m, n), in0=f32(n - 1), out0=f32(m)),
    "call bicg p of m": lambda: mep.make_call(mep.MEP_OP_BICG, f32(m, n), in0=f32(m), in1=f32(m),
                                              out0=f32(n), out1=f32(m)),
    "call ata_x t fp64": lambda: mep.make_call(mep.MEP_OP_ATA_X, f32(m, n), in0=f32(n), out0=f32(n),
                                               out1=f64(m)),
    "call axpby no B shape": lambda: mep.make_call(mep.MEP_OP_AXPBY_MV, f32(m, n), in0=f32(n), out0=f32(m),
                                                   B=f32(m, n + 1)),
    "call gemver Ahat short": lambda: mep.make_call(mep.MEP_OP_GEMVER, f32(m, n), in0=f32(m), in1=f32(n),
                                                    in2=f32(m), in3=f32(n), in4=f32(m), in5=f32(n),
                                                    out0=f32(n), out1=f32(m), out2=f32(m * n - 1)),
    "call matvec stray in1": lambda: mep.make_call(mep.MEP_OP_MATVEC, f32(m, n), in0=f32(n), in1=f32(n),
                                                   out0=f32(m)),
    "call reduce out of 2": lambda: mep.make_call(mep.MEP_OP_REDUCE_SUM, f32(n), out0=f32(2)),
    "call vector_add short b": lambda: mep.make_call(mep.MEP_OP_VECTOR_ADD, f32(n), in1=f32(n - 1),
                                                     out0=f32(n)),
}


@pytest.mark.parametrize("name", sorted(BAD_CALLS))
def test_bad_tensor_raises_before_the_c_abi(name):
    with pytest.raises(ValueError) as e:
        BAD_CALLS[name]()
    assert "GPU" not in str(e.value), f"{name}: refused for the device, not for the bad tensor"


def test_unsupported_dtype_raises():
    with pytest.raises(TypeError):
        mep.mep_matvec(torch.zeros(m, n, dtype=torch.float16), torch.zeros(n, dtype=torch.float16))


GOOD_HOST_CALLS = {
    "matvec": lambda: mep.mep_matvec(f32(m, n), f32(n)),
    "bicg": lambda: mep.mep_matvec_t(f32(m, n), f32(m), p=f32(n)),
    "ata_x": lambda: mep.mep_ata_x(f64(m, n), f64(n), t=f64(m)),
    "axpby_mv": lambda: mep.mep_axpby_mv(1.5, f32(m, n), 1.2, f32(m, n), f32(n)),
    "gemver": lambda: mep.mep_gemver(1.0, 1.0, f32(m, n), f32(m), f32(n), f32(m), f32(n), f32(m), f32(n)),
    "reduce_sum": lambda: mep.mep_reduce_sum(f32(n)),
    "vector_add": lambda: mep.mep_vector_add(f32(n), f32(n)),
}


@pytest.mark.parametrize("name", sorted(GOOD_HOST_CALLS))
def test_host_tensors_are_refused(name):
    with pytest.raises(ValueError, match="GPU"):
        GOOD_HOST_CALLS[name]()
