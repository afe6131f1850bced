"""GPU parity of the entry points with gates per (key slot, value channel)
(kla_forward_pc_ou, kla_backward_pc_ou, kla_decode_step_pc_ou): Algorithm 1's
Abar, Pbar : (N, D) from OU parameters a, p, delta [H, dk, dv], with the observation
precision per value channel, against the fp64 oracle's per-(n, d) mode.

Small shapes are compared over whole tensors; the language-model shape
(B8 T2048 H16 d128 bf16) runs at full size, with the per-token outputs compared on
sampled (batch, head) sequences and the parameter gradients of two whole heads
(every batch row) -- sums over (b, t), judged against the mass of their terms.
"""
import numpy as np
import pytest

import kla_inputs as K
import oracle
from kla_testutil import TOL, bits_to_torch, log, rel_err, rel_err_sum, to_np, to_torch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
NAMES = ("q", "k", "v", "rc")


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
    e = rel_err_sum(got, ref, mass)
    report.append(f"{name}={e:.2e}(plain {rel_err(got, ref):.1e})")
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert e <= tol, f"{name}: rel err {e:.3e} > {tol:.0e}"


def _f32(a):
    return torch.tensor(np.asarray(a), dtype=torch.float32, device=DEV)


def _case(B, T, H, dk, dv, dtype, seed, dist):
    w = K.Workload(0, "custom", B, T, H, dk, dv, dtype, dist, False)
    return K.full(w, names=NAMES + ("dy",), seed=seed)


def _ou(H, dk, dv, seed):
    P = K.ou_params(H, dk, seed, dv=dv)
    return {n: _f32(P[n]) for n in P}, {n: P[n].astype(np.float64) for n in P}


SMALL = [  # B, T, H, dk, dv, dtype, dist
    (2, 100, 3, 16, 16, "f32", "c0"),
    (1, 77, 2, 32, 64, "f32", "lm"),
    (2, 41, 1, 128, 16, "f32", "lm"),
    (2, 130, 2, 64, 32, "bf16", "lm"),
    (1, 70, 2, 128, 128, "bf16", "lm"),
    (1, 33, 1, 16, 128, "bf16", "c0"),
]


@pytest.mark.parametrize("B,T,H,dk,dv,dtype,dist", SMALL)
def test_pc_ou_forward_backward_small(kla, B, T, H, dk, dv, dtype, dist):
    case = _case(B, T, H, dk, dv, dtype, seed=T + dk, dist=dist)
    P, Pd = _ou(H, dk, dv, seed=dv)
    g = np.random.default_rng(T)
    q32 = lambda a: a.astype(np.float32).astype(np.float64)
    lam0, eta0 = q32(0.5 + g.random((B, H, dk, dv))), q32(g.standard_normal((B, H, dk, dv)))
    dlamT, detaT = q32(g.standard_normal((B, H, dk, dv))), q32(g.standard_normal((B, H, dk, dv)))
    dyvar = q32(g.standard_normal((B, T, H, dv)))
    log(f"pc ou small B{B} T{T} H{H} dk{dk} dv{dv} {dtype}")
    x = {n: to_torch(case[n], dtype, DEV) for n in NAMES + ("dy",)}
    out = kla.kla_forward_pc_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["rc"], _f32(lam0), _f32(eta0),
                                want_var=True, save=True)
    args = (x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["rc"], _f32(lam0), _f32(eta0), x["dy"],
            _f32(dlamT), _f32(detaT))
    gr = kla.kla_backward_pc_ou(*args, saved=out["saved"], dyvar=_f32(dyvar))
    gr2 = kla.kla_backward_pc_ou(*args, dyvar=_f32(dyvar))
    torch.cuda.synchronize()
    ref = oracle.forward_ou_nd(case["q"], case["k"], case["v"], Pd["a"], Pd["p"], Pd["delta"], case["rc"], lam0,
                               eta0)
    rg = oracle.backward_ou_nd(case["q"], case["k"], case["v"], Pd["a"], Pd["p"], Pd["delta"], case["rc"], lam0,
                               eta0, case["dy"], dlamT, detaT, dyvar)
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
    for n in ("dq", "dk", "dv", "dr", "da", "dp", "ddelta", "dlam0", "deta0"):
        assert torch.equal(gr[n], gr2[n]), f"{n} differs between saved and recomputed context"
    log("  " + " ".join(rep))


def test_pc_ou_decode_steps_equal_forward(kla):
    B, T, H, dk, dv = 3, 12, 2, 32, 16
    case = _case(B, T, H, dk, dv, "f32", seed=8, dist="lm")
    P, _ = _ou(H, dk, dv, seed=3)
    x = {n: to_torch(case[n], "f32", DEV) for n in NAMES}
    log("pc ou decode vs forward")
    full = kla.kla_forward_pc_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["rc"], want_var=True)
    lam = torch.ones(B, H, dk, dv, device=DEV)
    eta = torch.zeros(B, H, dk, dv, device=DEV)
    for t in range(T):
        sl = {n: x[n][:, t].contiguous() for n in NAMES}
        st = kla.kla_decode_step_pc_ou(sl["q"], sl["k"], sl["v"], P["a"], P["p"], P["delta"], sl["rc"], lam, eta,
                                       want_var=True)
        # the decode step stores the fp32 belief after every token, the forward carries it in fp64
        torch.testing.assert_close(st["y"], full["y"][:, t], rtol=1e-5, atol=1e-6)
        torch.testing.assert_close(st["yvar"], full["yvar"][:, t], rtol=1e-5, atol=1e-6)
    torch.testing.assert_close(lam, full["lamT"], rtol=1e-5, atol=1e-6)
    torch.testing.assert_close(eta, full["etaT"], rtol=1e-5, atol=1e-6)


def test_pc_ou_autograd_wrapper(kla):
    B, T, H, dk, dv = 2, 30, 1, 16, 16
    case = _case(B, T, H, dk, dv, "f32", seed=4, dist="c0")
    P, Pd = _ou(H, dk, dv, seed=4)
    leaves = {n: P[n].clone().requires_grad_(True) for n in P}
    x = {n: to_torch(case[n], "f32", DEV).requires_grad_(True) for n in NAMES}
    log("pc ou autograd")
    y, _, _ = kla.kla_filter_pc_ou(x["q"], x["k"], x["v"], leaves["a"], leaves["p"], leaves["delta"], x["rc"])
    (y * to_torch(case["dy"], "f32", DEV)).sum().backward()
    rg = oracle.backward_ou_nd(case["q"], case["k"], case["v"], Pd["a"], Pd["p"], Pd["delta"], case["rc"], None,
                               None, case["dy"])
    for n, gn in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("rc", "dr")):
        assert rel_err(to_np(x[n].grad), rg[gn]) <= TOL["f32"], n
    for n, gn in (("a", "da"), ("p", "dp"), ("delta", "ddelta")):
        assert rel_err_sum(to_np(leaves[n].grad), rg[gn], rg["mass_" + gn]) <= TOL["f32"], n


def test_pc_ou_check_mode_rejects_bad_parameters(kla, monkeypatch):
    B, T, H, dk, dv = 1, 8, 1, 16, 16
    case = _case(B, T, H, dk, dv, "f32", seed=5, dist="c0")
    P, _ = _ou(H, dk, dv, seed=5)
    P["delta"][0, 3, 7] = -1.0
    x = {n: to_torch(case[n], "f32", DEV) for n in NAMES}
    log("pc ou check mode")
    monkeypatch.setenv("KLA_CHECK", "1")
    with pytest.raises(kla.KLAError) as ei:
        kla.kla_forward_pc_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["rc"])
    assert ei.value.status == 6


def test_pc_ou_lm_layer_full_size(kla):
    """B8 T2048 H16 d128 bf16, r per value channel, OU parameters [16, 128, 128]."""
    w = K.Workload(2, "lm_layer_1p3b_bf16", 8, 2048, 16, 128, 128, "bf16", "lm", True)
    log(f"pc ou lm layer B{w.B} T{w.T} H{w.H} d{w.dk}: generating inputs")
    bits = K.full(w, names=NAMES + ("dy",), as_bits=True)
    x = {n: bits_to_torch(bits[n], DEV) for n in bits}
    del bits
    P, Pd = _ou(w.H, w.dk, w.dv, seed=w.cid)
    log("pc ou lm layer: forward and backward on GPU")
    out = kla.kla_forward_pc_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["rc"], want_var=True,
                                save=True)
    gr = kla.kla_backward_pc_ou(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["rc"], None, None, x["dy"],
                                saved=out["saved"], want_init_grads=False)
    torch.cuda.synchronize()
    tol = TOL[w.dtype]
    rep = []
    for h in (5, w.H - 1):
        pairs = [(b, h) for b in range(w.B)]
        log(f"pc ou lm layer: oracle on head {h}, every batch row")
        sl = K.pairs_slice(w, pairs, names=NAMES + ("dy",))
        hp = {n: Pd[n][h:h + 1] for n in Pd}
        ref = oracle.forward_ou_nd(sl["q"], sl["k"], sl["v"], hp["a"], hp["p"], hp["delta"], sl["rc"])
        rg = oracle.backward_ou_nd(sl["q"], sl["k"], sl["v"], hp["a"], hp["p"], hp["delta"], sl["rc"], None, None,
                                   sl["dy"])
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
    log("  pc ou lm layer: " + " ".join(rep))
