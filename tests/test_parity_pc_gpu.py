"""GPU parity of the per-channel-precision entry points (kla_forward_pc,
kla_backward_pc, kla_decode_step_pc) against the fp64 oracle, which runs every (n, d) filter
with its own precision (r [B, T, H, dv], beliefs [B, H, dk, dv]).

Small shapes are compared over whole tensors; the language-model shape
(B8 T2048 H16 d128 bf16, r drawn per value channel) runs at full size and is
compared on sampled (batch, head) sequences.
"""
import numpy as np
import pytest

import kla_inputs as K
import oracle
from kla_testutil import TOL, bits_to_torch, log, rel_err, to_np, to_torch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
NAMES = ("q", "k", "v", "a", "p", "rc")


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


def _f32(a):
    return torch.tensor(np.asarray(a), dtype=torch.float32, device=DEV)


def _case(B, T, H, dk, dv, dtype, seed, dist):
    w = K.Workload(0, "custom", B, T, H, dk, dv, dtype, dist, False)
    return K.full(w, names=NAMES, seed=seed)


PC_SMALL = [  # B, T, H, dk, dv, dtype, dist
    (2, 100, 3, 16, 16, "f32", "c0"),
    (1, 77, 2, 32, 64, "f32", "lm"),
    (3, 41, 1, 128, 16, "f32", "lm"),
    (2, 130, 2, 64, 32, "bf16", "lm"),
    (1, 70, 2, 128, 128, "bf16", "lm"),
    (1, 33, 1, 16, 128, "bf16", "c0"),
]


@pytest.mark.parametrize("B,T,H,dk,dv,dtype,dist", PC_SMALL)
@pytest.mark.parametrize("init", [False, True])
def test_pc_forward_small(kla, B, T, H, dk, dv, dtype, dist, init):
    case = _case(B, T, H, dk, dv, dtype, seed=T * 5 + dk, dist=dist)
    lam0 = eta0 = None
    if init:
        g = np.random.default_rng(T)
        lam0 = (0.5 + g.random((B, H, dk, dv))).astype(np.float32).astype(np.float64)
        eta0 = g.standard_normal((B, H, dk, dv)).astype(np.float32).astype(np.float64)
    log(f"pc forward B{B} T{T} H{H} dk{dk} dv{dv} {dtype} init={init}")
    x = {n: to_torch(case[n], dtype, DEV) for n in NAMES}
    out = kla.kla_forward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"],
                             None if lam0 is None else _f32(lam0), None if eta0 is None else _f32(eta0),
                             want_var=True)
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["rc"], lam0, eta0)
    tol = TOL[dtype]
    rep = []
    _check("y", to_np(out["y"]), K.quantise(ref["y"], dtype), tol, rep)
    _check("yvar", to_np(out["yvar"]), ref["yvar"], TOL["f32"], rep)
    _check("lamT", to_np(out["lamT"]), ref["lamT"], TOL["f32"], rep)
    _check("etaT", to_np(out["etaT"]), ref["etaT"], TOL["f32"], rep)
    assert np.all(to_np(out["lamT"]) > 0) and np.all(to_np(out["yvar"]) > 0)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("B,T,H,dk,dv,dtype,dist", PC_SMALL)
def test_pc_backward_small(kla, B, T, H, dk, dv, dtype, dist):
    case = _case(B, T, H, dk, dv, dtype, seed=T * 3 + dv, dist=dist)
    g = np.random.default_rng(T + 11)
    q32 = lambda x: x.astype(np.float32).astype(np.float64)
    lam0 = q32(0.5 + g.random((B, H, dk, dv)))
    eta0 = q32(g.standard_normal((B, H, dk, dv)))
    dlamT = q32(g.standard_normal((B, H, dk, dv)))
    detaT = q32(g.standard_normal((B, H, dk, dv)))
    dyvar = q32(g.standard_normal((B, T, H, dv)))
    dy = K.quantise(g.standard_normal((B, T, H, dv)), dtype)
    log(f"pc backward B{B} T{T} H{H} dk{dk} dv{dv} {dtype}")
    x = {n: to_torch(case[n], dtype, DEV) for n in NAMES}
    dyt = to_torch(dy, dtype, DEV)
    out = kla.kla_forward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], _f32(lam0), _f32(eta0), save=True)
    gr = kla.kla_backward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], _f32(lam0), _f32(eta0), dyt,
                             _f32(dlamT), _f32(detaT), saved=out["saved"], dyvar=_f32(dyvar))
    gr2 = kla.kla_backward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], _f32(lam0), _f32(eta0), dyt,
                              _f32(dlamT), _f32(detaT), dyvar=_f32(dyvar))
    torch.cuda.synchronize()
    ref = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["rc"], lam0, eta0, dy,
                          dlamT, detaT, dyvar=dyvar)
    tol = TOL[dtype]
    rep = []
    for n in ("dq", "dk", "dv", "da", "dp", "dr", "dlam0", "deta0"):
        _check(n, to_np(gr[n]), ref[n], tol, rep)
    for n in ("dq", "dk", "dv", "da", "dp", "dr", "dlam0", "deta0"):
        assert torch.equal(gr[n], gr2[n]), f"{n} differs between saved and recomputed context"
    log("  " + " ".join(rep))


def test_pc_empty_sequence(kla):
    B, H, dk, dv = 2, 2, 32, 16
    g = np.random.default_rng(1)
    lam0 = (0.5 + g.random((B, H, dk, dv))).astype(np.float32)
    eta0 = g.standard_normal((B, H, dk, dv)).astype(np.float32)
    for tdt in (torch.float32, torch.bfloat16):
        e = lambda *s: torch.empty(s, dtype=tdt, device=DEV)
        log(f"pc edge T=0 {tdt}")
        out = kla.kla_forward_pc(e(B, 0, H, dk), e(B, 0, H, dk), e(B, 0, H, dv), e(B, 0, H, dk), e(B, 0, H, dk),
                                 e(B, 0, H, dv), _f32(lam0), _f32(eta0))
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_np(out["lamT"]), lam0)
        np.testing.assert_array_equal(to_np(out["etaT"]), eta0)


def test_pc_decode_steps_equal_forward(kla):
    S, H, dk, dv, steps = 6, 2, 64, 32, 5
    case = _case(S, steps, H, dk, dv, "f32", seed=23, dist="lm")
    g = np.random.default_rng(2)
    lam = (0.5 + g.random((S, H, dk, dv))).astype(np.float32).astype(np.float64)
    eta = g.standard_normal((S, H, dk, dv)).astype(np.float32).astype(np.float64)
    lam_d, eta_d = _f32(lam), _f32(eta)
    rep = []
    for t in range(steps):
        x = {n: to_torch(np.ascontiguousarray(case[n][:, t]), "f32", DEV) for n in NAMES}
        log(f"pc decode step {t}")
        out = kla.kla_decode_step_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], lam_d, eta_d, want_var=True)
        torch.cuda.synchronize()
        ref = oracle.decode_step(case["q"][:, t], case["k"][:, t], case["v"][:, t], case["a"][:, t],
                                 case["p"][:, t], case["rc"][:, t], lam, eta)
        lam, eta = ref["lam"], ref["eta"]
        for n, got, want in (("y", out["y"], ref["y"]), ("yvar", out["yvar"], ref["yvar"]),
                             ("lam", lam_d, lam), ("eta", eta_d, eta)):
            _check(f"{n}{t}", to_np(got), want, TOL["f32"], rep)
    log("  pc decode: " + " ".join(rep))


def test_pc_check_mode_rejects_bad_channel_precision(kla, monkeypatch):
    monkeypatch.setenv("KLA_CHECK", "1")
    B, T, H, dk, dv = 1, 20, 2, 32, 64
    case = _case(B, T, H, dk, dv, "f32", seed=4, dist="lm")
    x = {n: to_torch(case[n], "f32", DEV) for n in NAMES}
    kla.kla_forward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"])   # in the domain
    bad = x["rc"].clone()
    bad[0, T - 1, H - 1, dv - 1] = -1.0   # the last element: the check must cover every channel
    log("pc check mode: r < 0 in the last channel")
    with pytest.raises(kla.KLAError, match="NUMERIC"):
        kla.kla_forward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], bad)


def test_pc_lm_layer_full_size(kla):
    """B8 T2048 H16 d128 bf16 with r per value channel, sampled sequences."""
    w = K.WORKLOADS[2]
    log(f"pc lm layer B{w.B} T{w.T} H{w.H} d{w.dk}: generating inputs")
    bits = K.full(w, names=NAMES, as_bits=True)
    x = {n: bits_to_torch(bits[n], DEV) for n in bits}
    del bits
    dyb = bits_to_torch(K.full(w, names=("dy",), as_bits=True)["dy"], DEV)
    log("pc lm layer: forward and backward on GPU")
    out = kla.kla_forward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], want_var=True, save=True)
    gr = kla.kla_backward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], None, None, dyb,
                             saved=out["saved"], want_init_grads=False)
    torch.cuda.synchronize()
    g = np.random.default_rng(0)
    pairs = {(0, 0), (w.B - 1, w.H - 1)}
    while len(pairs) < 6:
        pairs.add((int(g.integers(w.B)), int(g.integers(w.H))))
    pairs = sorted(pairs)
    log(f"pc lm layer: oracle on pairs {pairs}")
    sl = K.pairs_slice(w, pairs, names=NAMES + ("dy",))
    ref = oracle.forward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["rc"])
    rg = oracle.backward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["rc"], None, None, sl["dy"])
    bi = [b for b, _ in pairs]
    hi = [h for _, h in pairs]
    tol = TOL[w.dtype]
    rep = []
    _check("y", to_np(out["y"][bi, :, hi]), K.quantise(ref["y"][:, :, 0], w.dtype), tol, rep)
    _check("yvar", to_np(out["yvar"][bi, :, hi]), ref["yvar"][:, :, 0], tol, rep)
    _check("lamT", to_np(out["lamT"][bi, hi]), ref["lamT"][:, 0], tol, rep)
    _check("etaT", to_np(out["etaT"][bi, hi]), ref["etaT"][:, 0], tol, rep)
    for n in ("dq", "dk", "dv", "da", "dp", "dr"):
        _check(n, to_np(gr[n][bi, :, hi]), rg[n][:, :, 0], tol, rep)
        assert torch.isfinite(gr[n].float()).all(), n
    assert torch.all(out["lamT"] > 0) and torch.all(out["yvar"] > 0)
    assert torch.isfinite(out["y"].float()).all()
    log("  pc lm layer: " + " ".join(rep))
