"""GPU parity of the block scaffolding (causal conv1d + SiLU, RMS QK-norm, SiLU
gate; forward and backward) against the fp64 oracle in oracle/block.py, on
small ragged shapes and at the LM-layer shape (B8 T2048, C = H dk = 2048,
rows = B T H of n = 128)."""
import numpy as np
import pytest

import kla_inputs as K
from oracle import block as OB
from kla_testutil import TOL, log, rel_err, to_np, to_torch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def kla():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_10743_amd as lib
    lib._load()
    return lib


def _check(name, got, ref, tol, report):
    e = rel_err(got, ref)
    report.append(f"{name}={e:.2e}")
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert e <= tol, f"{name}: rel err {e:.3e} > {tol:.0e}"


def _f32(a):
    return torch.tensor(np.asarray(a), dtype=torch.float32, device=DEV)


def _q(x, dtype):
    return K.quantise(x, dtype)


@pytest.mark.parametrize("B,T,C,dtype,with_bias", [
    (2, 100, 64, "f32", True), (1, 3, 16, "f32", False), (3, 130, 40, "bf16", True),
    (2, 65, 128, "bf16", False), (1, 1, 8, "bf16", True), (2, 200, 48, "f32", True)])
def test_conv_silu(kla, B, T, C, dtype, with_bias):
    g = np.random.default_rng(T + C)
    x = _q(g.standard_normal((B, T, C)), dtype)
    du = _q(g.standard_normal((B, T, C)), dtype)
    w = (0.5 * g.standard_normal((C, 4))).astype(np.float32).astype(np.float64)
    bias = g.standard_normal(C).astype(np.float32).astype(np.float64) if with_bias else None
    log(f"conv B{B} T{T} C{C} {dtype} bias={with_bias}")
    xt, dut = to_torch(x, dtype, DEV), to_torch(du, dtype, DEV)
    bt = None if bias is None else _f32(bias)
    u = kla.kla_conv_silu_forward(xt, _f32(w), bt)
    dx, dw, db = kla.kla_conv_silu_backward(xt, _f32(w), bt, dut)
    torch.cuda.synchronize()
    ref_u = OB.conv_silu_forward(x, w, bias)
    rdx, rdw, rdb = OB.conv_silu_backward(x, w, bias, du)
    tol = TOL[dtype]
    rep = []
    _check("u", to_np(u), _q(ref_u, dtype), tol, rep)
    _check("dx", to_np(dx), _q(rdx, dtype), tol, rep)
    _check("dw", to_np(dw), rdw, TOL["f32"] if dtype == "f32" else 1e-3, rep)
    if with_bias:
        _check("db", to_np(db), rdb, TOL["f32"] if dtype == "f32" else 1e-3, rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("rows,n,dtype", [(37, 16, "f32"), (300, 32, "bf16"), (513, 64, "f32"), (1000, 128, "bf16"),
                                          (5, 128, "f32")])
def test_qk_norm(kla, rows, n, dtype):
    g = np.random.default_rng(rows + n)
    x = _q(3.0 * g.standard_normal((rows, n)), dtype)
    dout = _q(g.standard_normal((rows, n)), dtype)
    w = (1.0 + 0.1 * g.standard_normal(n)).astype(np.float32).astype(np.float64)
    eps = 1e-6
    log(f"qk norm rows{rows} n{n} {dtype}")
    xt = to_torch(x, dtype, DEV)
    out, rstd = kla.kla_qk_norm_forward(xt, _f32(w), eps)
    dx, dw = kla.kla_qk_norm_backward(xt, _f32(w), rstd, to_torch(dout, dtype, DEV))
    torch.cuda.synchronize()
    ref, rr = OB.rmsnorm_forward(x, w, eps)
    rdx, rdw = OB.rmsnorm_backward(x, w, eps, dout)
    tol = TOL[dtype]
    rep = []
    _check("out", to_np(out), _q(ref, dtype), tol, rep)
    _check("rstd", to_np(rstd), rr, TOL["f32"], rep)
    _check("dx", to_np(dx), _q(rdx, dtype), tol, rep)
    _check("dw", to_np(dw), rdw, TOL["f32"] if dtype == "f32" else 1e-3, rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("n,dtype", [(8, "bf16"), (1000, "f32"), (4096 + 64, "bf16"), (123456, "f32")])
def test_gate(kla, n, dtype):
    g = np.random.default_rng(n)
    y, z, do = (_q(g.standard_normal(n) * s, dtype) for s in (1.0, 3.0, 1.0))
    log(f"gate n{n} {dtype}")
    yt, zt = to_torch(y, dtype, DEV), to_torch(z, dtype, DEV)
    out = kla.kla_gate_forward(yt, zt)
    dy, dz = kla.kla_gate_backward(yt, zt, to_torch(do, dtype, DEV))
    torch.cuda.synchronize()
    rdy, rdz = OB.gate_backward(y, z, do)
    tol = TOL[dtype]
    rep = []
    _check("out", to_np(out), _q(OB.gate_forward(y, z), dtype), tol, rep)
    _check("dy", to_np(dy), _q(rdy, dtype), tol, rep)
    _check("dz", to_np(dz), _q(rdz, dtype), tol, rep)
    log("  " + " ".join(rep))


def test_conv_empty_sequence(kla):
    x = torch.empty((2, 0, 16), dtype=torch.bfloat16, device=DEV)
    w = _f32(np.ones((16, 4)))
    b = _f32(np.ones(16))
    u = kla.kla_conv_silu_forward(x, w, b)
    dx, dw, db = kla.kla_conv_silu_backward(x, w, b, torch.empty_like(x))
    torch.cuda.synchronize()
    assert u.numel() == 0 and dx.numel() == 0
    assert torch.count_nonzero(dw) == 0 and torch.count_nonzero(db) == 0


def test_scaffolding_lm_shape(kla):
    """B8 T2048 H16 dk128 bf16: the conv over C = H dk channels, the norm over
    the B T H rows of q, the gate over the layer output; whole tensors."""
    B, T, H, d = 8, 2048, 16, 128
    C = H * d
    g = np.random.default_rng(42)
    log("scaffolding lm shape: inputs")
    x = _q(g.standard_normal((B, T, C)), "bf16")
    du = _q(g.standard_normal((B, T, C)), "bf16")
    w = (0.5 * g.standard_normal((C, 4))).astype(np.float32).astype(np.float64)
    bias = g.standard_normal(C).astype(np.float32).astype(np.float64)
    xt, dut = to_torch(x, "bf16", DEV), to_torch(du, "bf16", DEV)
    u = kla.kla_conv_silu_forward(xt, _f32(w), _f32(bias))
    dx, dw, db = kla.kla_conv_silu_backward(xt, _f32(w), _f32(bias), dut)
    rows = x.reshape(B * T * H, d)
    nw = (1.0 + 0.1 * g.standard_normal(d)).astype(np.float32).astype(np.float64)
    out, rstd = kla.kla_qk_norm_forward(xt.view(B * T * H, d), _f32(nw), 1e-6)
    ndx, ndw = kla.kla_qk_norm_backward(xt.view(B * T * H, d), _f32(nw), rstd, dut.view(B * T * H, d))
    gout = kla.kla_gate_forward(xt, dut)
    torch.cuda.synchronize()
    log("scaffolding lm shape: oracle")
    rep = []
    tol = TOL["bf16"]
    _check("conv_u", to_np(u), _q(OB.conv_silu_forward(x, w, bias), "bf16"), tol, rep)
    rdx, rdw, rdb = OB.conv_silu_backward(x, w, bias, du)
    _check("conv_dx", to_np(dx), _q(rdx, "bf16"), tol, rep)
    _check("conv_dw", to_np(dw), rdw, 1e-3, rep)
    _check("conv_db", to_np(db), rdb, 1e-3, rep)
    ref, _ = OB.rmsnorm_forward(rows, nw, 1e-6)
    _check("norm_out", to_np(out), _q(ref, "bf16"), tol, rep)
    rndx, rndw = OB.rmsnorm_backward(rows, nw, 1e-6, du.reshape(B * T * H, d))
    _check("norm_dx", to_np(ndx), _q(rndx, "bf16"), tol, rep)
    _check("norm_dw", to_np(ndw), rndw, 1e-3, rep)
    _check("gate", to_np(gout), _q(OB.gate_forward(x, du), "bf16"), tol, rep)
    log("  scaffolding: " + " ".join(rep))
