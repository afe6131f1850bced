"""GPU parity of the OU-gated entry points (kla_forward_ou, kla_backward_ou,
kla_decode_step_ou) against the fp64 oracle's ``*_ou`` functions.

The gates come from time-invariant OU parameters a, p, delta [H, dk] (Sec. 4.1,
eq. discretisation); the per-token tensors are drawn as in the other parity
tests.  Small shapes are compared over whole tensors, on both the chunked MFMA
path (bf16, dk >= 32) and the token-recurrent path; the language-model shape
(B8 T2048 H16 d128 bf16) runs at full size and is compared on sampled
sequences, and on whole heads for the parameter gradients, which sum over every
batch row.
"""
import os

import numpy as np
import pytest

import kla_inputs as K
import oracle
from kla_testutil import TOL, bits_to_torch, log, rel_err, rel_err_sum, to_np, to_torch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOKEN_NAMES = ("q", "k", "v", "r", "dy")


@pytest.fixture(scope="module")
def kla():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_10743_amd as lib
    lib._load()
    return lib


def _check(name, got, ref, tol, report):
    e = rel_err(got, ref)
    report.append(f"{name}={e:.2e}(rms-rel {rel_err(got, ref, 1.0):.1e})")
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert e <= tol, f"{name}: rel err {e:.3e} > {tol:.0e}"


def _check_sum(name, got, ref, mass, tol, report):
    """Parameter gradients: sums over (b, t), judged against the mass of their terms."""
    e = rel_err_sum(got, ref, mass)
    report.append(f"{name}={e:.2e}(plain {rel_err(got, ref):.1e})")
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert e <= tol, f"{name}: rel err {e:.3e} > {tol:.0e}"


def _f32(a):
    return torch.tensor(np.asarray(a), dtype=torch.float32, device=DEV)


def _ou(H, dk, seed):
    """OU parameters as float32 (device) and their exact float64 widening (oracle)."""
    P = K.ou_params(H, dk, seed)
    return ({n: _f32(P[n]) for n in ("a", "p", "delta")},
            {n: P[n].astype(np.float64) for n in ("a", "p", "delta")})


def _belief(B, H, dk, dv, seed):
    g = np.random.default_rng(seed)
    lam0 = (0.5 + g.random((B, H, dk))).astype(np.float32).astype(np.float64)
    eta0 = g.standard_normal((B, H, dk, dv)).astype(np.float32).astype(np.float64)
    return lam0, eta0


OU_SMALL = [  # B, T, H, dk, dv, dtype, dist
    (2, 100, 3, 16, 16, "f32", "c0"),
    (1, 77, 2, 32, 64, "f32", "lm"),
    (2, 95, 2, 32, 32, "f32", "lm"),
    (1, 64, 3, 32, 16, "f32", "c0"),
    (2, 33, 1, 16, 32, "f32", "lm"),
    (1, 33, 2, 16, 128, "bf16", "c0"),
    (2, 130, 2, 64, 32, "bf16", "lm"),
    (1, 200, 2, 128, 128, "bf16", "lm"),
    (1, 31, 1, 64, 128, "bf16", "lm"),
    (3, 161, 1, 32, 32, "bf16", "c0"),
]


@pytest.mark.parametrize("B,T,H,dk,dv,dtype,dist", OU_SMALL)
def test_ou_forward_backward_small(kla, B, T, H, dk, dv, dtype, dist):
    case = K.random_case(B, T, H, dk, dv, dtype, seed=T * 13 + dk, dist=dist)
    P, Pd = _ou(H, dk, seed=T + dv)
    lam0, eta0 = _belief(B, H, dk, dv, T + 2)
    g = np.random.default_rng(T + 3)
    dlamT = g.standard_normal((B, H, dk)).astype(np.float32).astype(np.float64)
    detaT = g.standard_normal((B, H, dk, dv)).astype(np.float32).astype(np.float64)
    dyvar = g.standard_normal((B, T, H)).astype(np.float32).astype(np.float64)
    log(f"ou small B{B} T{T} H{H} dk{dk} dv{dv} {dtype}")
    x = {n: to_torch(case[n], dtype, DEV) for n in TOKEN_NAMES}
    out = kla.kla_forward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], _f32(lam0), _f32(eta0),
                             want_var=True, save=True)
    gr = kla.kla_backward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], _f32(lam0), _f32(eta0),
                             x["dy"], _f32(dlamT), _f32(detaT), saved=out["saved"], dyvar=_f32(dyvar))
    # the backward without a saved context recomputes it and must agree bit for bit
    gr2 = kla.kla_backward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], _f32(lam0),
                              _f32(eta0), x["dy"], _f32(dlamT), _f32(detaT), dyvar=_f32(dyvar))
    torch.cuda.synchronize()
    ref = oracle.forward_ou(case["q"], case["k"], case["v"], Pd["a"], Pd["p"], Pd["delta"], case["r"], lam0, eta0)
    rg = oracle.backward_ou(case["q"], case["k"], case["v"], Pd["a"], Pd["p"], Pd["delta"], case["r"], lam0, eta0,
                            case["dy"], dlamT, detaT, dyvar=dyvar, with_mass=True)
    tol = TOL[dtype]
    rep = []
    _check("y", to_np(out["y"]), K.quantise(ref["y"], dtype), tol, rep)
    _check("yvar", to_np(out["yvar"]), ref["yvar"], TOL["f32"], rep)
    _check("lamT", to_np(out["lamT"]), ref["lamT"], TOL["f32"], rep)
    _check("etaT", to_np(out["etaT"]), ref["etaT"], tol if dtype == "bf16" else TOL["f32"], rep)
    for n in ("dq", "dk", "dv", "dr", "dlam0", "deta0"):
        _check(n, to_np(gr[n]), rg[n], tol, rep)
    for n in ("da", "dp", "ddelta"):
        _check_sum(n, to_np(gr[n]), rg[n], rg["mass_" + n], tol, rep)
    for n in ("dq", "dk", "dv", "dr", "da", "dp", "ddelta"):
        assert torch.equal(gr[n], gr2[n]), f"{n} differs between saved and recomputed context"
    assert np.all(to_np(out["lamT"]) > 0) and np.all(to_np(out["yvar"]) > 0)
    log("  " + " ".join(rep))


def test_ou_empty_sequence(kla):
    """T = 0: the belief passes through, its gradients pass back, the parameter gradients are zero."""
    B, H, dk, dv = 2, 2, 32, 16
    for dtype in ("f32", "bf16"):
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        P, Pd = _ou(H, dk, seed=1)
        lam0, eta0 = _belief(B, H, dk, dv, 4)
        e = lambda *s: torch.empty(s, dtype=tdt, device=DEV)
        q, k, v, r, dy = e(B, 0, H, dk), e(B, 0, H, dk), e(B, 0, H, dv), e(B, 0, H), e(B, 0, H, dv)
        log(f"ou edge T=0 {dtype}")
        out = kla.kla_forward_ou(q, k, v, P["a"], P["p"], P["delta"], r, _f32(lam0), _f32(eta0))
        gr = kla.kla_backward_ou(q, k, v, P["a"], P["p"], P["delta"], r, _f32(lam0), _f32(eta0), dy,
                                 _f32(np.ones((B, H, dk))), _f32(np.ones((B, H, dk, dv))))
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_np(out["lamT"]), lam0)
        np.testing.assert_array_equal(to_np(out["etaT"]), eta0)
        np.testing.assert_array_equal(to_np(gr["dlam0"]), np.ones((B, H, dk)))
        np.testing.assert_array_equal(to_np(gr["deta0"]), np.ones((B, H, dk, dv)))
        for n in ("da", "dp", "ddelta"):
            assert torch.count_nonzero(gr[n]) == 0, n


def test_ou_decode_steps(kla):
    S, H, dk, dv, steps = 5, 3, 32, 64, 4
    P, Pd = _ou(H, dk, seed=2)
    case = K.random_case(S, steps, H, dk, dv, "f32", seed=17, dist="lm")
    lam, eta = _belief(S, H, dk, dv, 6)
    lam_d, eta_d = _f32(lam), _f32(eta)
    rep = []
    for t in range(steps):
        x = {n: to_torch(np.ascontiguousarray(case[n][:, t]), "f32", DEV) for n in ("q", "k", "v", "r")}
        out = kla.kla_decode_step_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], lam_d, eta_d,
                                     want_var=True)
        torch.cuda.synchronize()
        ref = oracle.decode_step_ou(case["q"][:, t], case["k"][:, t], case["v"][:, t], Pd["a"], Pd["p"],
                                    Pd["delta"], case["r"][:, t], lam, eta)
        lam, eta = ref["lam"], ref["eta"]
        for n, got, want in (("y", out["y"], ref["y"]), ("yvar", out["yvar"], ref["yvar"]),
                             ("lam", lam_d, lam), ("eta", eta_d, eta)):
            _check(f"{n}{t}", to_np(got), want, TOL["f32"], rep)
    log("  ou decode: " + " ".join(rep))


def test_ou_check_mode_rejects_bad_parameters(kla, monkeypatch):
    monkeypatch.setenv("KLA_CHECK", "1")
    B, T, H, dk, dv = 1, 40, 2, 32, 32
    case = K.random_case(B, T, H, dk, dv, "bf16", seed=3, dist="lm")
    x = {n: to_torch(case[n], "bf16", DEV) for n in TOKEN_NAMES}
    P, _ = _ou(H, dk, seed=3)
    kla.kla_forward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"])   # in the domain
    for name, value in (("a", 0.0), ("delta", -1.0), ("p", float("nan"))):
        bad = dict(P)
        bad[name] = P[name].clone()
        bad[name][1, 5] = value
        log(f"ou check mode: {name} = {value}")
        with pytest.raises(kla.KLAError, match="NUMERIC"):
            kla.kla_forward_ou(x["q"], x["k"], x["v"], bad["a"], bad["p"], bad["delta"], x["r"])


def test_ou_autograd_wrapper(kla):
    B, T, H, dk, dv = 1, 70, 2, 64, 64
    case = K.random_case(B, T, H, dk, dv, "bf16", seed=21, dist="lm")
    x = {n: to_torch(case[n], "bf16", DEV) for n in TOKEN_NAMES}
    P, _ = _ou(H, dk, seed=21)
    leaves = {n: P[n].clone().requires_grad_(True) for n in ("a", "p", "delta")}
    y, yvar, lamT, etaT = kla.kla_filter_ou(x["q"], x["k"], x["v"], leaves["a"], leaves["p"], leaves["delta"],
                                            x["r"], want_var=True)
    gv = torch.randn(yvar.shape, generator=torch.Generator().manual_seed(4)).to(DEV)
    torch.autograd.backward([y, yvar], [x["dy"], gv])
    gr = kla.kla_backward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], None, None, x["dy"],
                             _f32(np.zeros((B, H, dk))), _f32(np.zeros((B, H, dk, dv))), dyvar=gv)
    torch.cuda.synchronize()
    for n, g in (("a", "da"), ("p", "dp"), ("delta", "ddelta")):
        assert torch.equal(leaves[n].grad, gr[g]), n


def test_ou_lm_layer_full_size(kla):
    """B8 T2048 H16 d128 bf16 with OU gates: sampled sequences for the per-token
    outputs, and two whole heads (all eight batch rows) for da, dp, ddelta."""
    w = K.WORKLOADS[2]
    log(f"ou lm layer B{w.B} T{w.T} H{w.H} d{w.dk}: generating inputs")
    bits = K.full(w, names=TOKEN_NAMES, as_bits=True)
    x = {n: bits_to_torch(bits[n], DEV) for n in bits}
    del bits
    P, Pd = _ou(w.H, w.dk, seed=w.cid)
    log("ou lm layer: forward and backward on GPU")
    out = kla.kla_forward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], want_var=True, save=True)
    gr = kla.kla_backward_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], None, None, x["dy"],
                             saved=out["saved"], want_init_grads=False)
    torch.cuda.synchronize()
    tol = TOL[w.dtype]
    rep = []
    for h in (3, w.H - 1):
        pairs = [(b, h) for b in range(w.B)]
        log(f"ou lm layer: oracle on head {h}, every batch row")
        sl = K.pairs_slice(w, pairs, names=TOKEN_NAMES)
        hp = {n: Pd[n][h:h + 1] for n in Pd}
        ref = oracle.forward_ou(sl["q"], sl["k"], sl["v"], hp["a"], hp["p"], hp["delta"], sl["r"])
        rg = oracle.backward_ou(sl["q"], sl["k"], sl["v"], hp["a"], hp["p"], hp["delta"], sl["r"], None, None,
                                sl["dy"], with_mass=True)
        bi = list(range(w.B))
        _check(f"y[h{h}]", to_np(out["y"][bi, :, h]), K.quantise(ref["y"][:, :, 0], w.dtype), tol, rep)
        _check(f"yvar[h{h}]", to_np(out["yvar"][bi, :, h]), ref["yvar"][:, :, 0], tol, rep)
        for n in ("dq", "dk", "dv", "dr"):
            _check(f"{n}[h{h}]", to_np(gr[n][bi, :, h]), rg[n][:, :, 0], tol, rep)
        for n in ("da", "dp", "ddelta"):
            _check_sum(f"{n}[h{h}]", to_np(gr[n][h:h + 1]), rg[n], rg["mass_" + n], tol, rep)
    for n in ("dq", "dk", "dv", "dr", "da", "dp", "ddelta"):
        assert torch.isfinite(gr[n].float()).all(), n
    assert torch.all(out["lamT"] > 0) and torch.all(out["yvar"] > 0)
    log("  ou lm layer: " + " ".join(rep))
