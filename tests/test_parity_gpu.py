"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small seeded shapes are compared element by element over whole tensors; the
five workloads run at their full sizes on the GPU and are compared on sampled
(batch, head) sequences, which the oracle computes on their own (every
(batch, head) pair is an independent filter).
"""
import os

import numpy as np
import pytest

import kla_inputs as K
import oracle
from kla_testutil import TOL, bits_to_torch, log, rel_err, to_np, to_torch

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
    report.append(f"{name}={e:.2e}(rms-rel {rel_err(got, ref, 1.0):.1e})")
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert e <= tol, f"{name}: rel err {e:.3e} > {tol:.0e}"


def _dev_inputs(case, dtype, names=K.NAMES + ("dy",)):
    return {n: to_torch(case[n], dtype, DEV) for n in names}


def _random_belief(B, H, dk, dv, seed):
    g = np.random.default_rng(seed)
    lam0 = 0.5 + g.random((B, H, dk))
    eta0 = g.standard_normal((B, H, dk, dv))
    return lam0.astype(np.float32).astype(np.float64), eta0.astype(np.float32).astype(np.float64)


SMALL = [  # B, T, H, dk, dv, dtype, dist
    (2, 100, 3, 16, 16, "f32", "c0"),
    (1, 77, 2, 32, 64, "f32", "c0"),
    (1, 65, 1, 128, 16, "f32", "lm"),
    (2, 130, 2, 64, 32, "bf16", "lm"),
    (1, 200, 2, 128, 128, "bf16", "lm"),
    (1, 33, 2, 16, 128, "bf16", "c0"),
    (3, 129, 2, 128, 128, "f32", "lm"),
    (2, 47, 2, 64, 64, "f32", "lm"),
    (1, 9, 1, 16, 32, "f32", "c0"),
    # chunked path at the other widths, partial chunks, a single short chunk, B*H not a multiple of 8
    (1, 97, 3, 32, 64, "bf16", "lm"),
    (2, 64, 1, 128, 32, "bf16", "lm"),
    (1, 31, 1, 64, 128, "bf16", "lm"),
    (3, 161, 1, 32, 32, "bf16", "c0"),
    # bf16 with dk >= 32 and dv = 16: chunked forward without a saved context, token-recurrent
    # backward (and forward, when the context is saved)
    (2, 70, 2, 64, 16, "bf16", "lm"),
    # chunked fp64 path (fp32 inputs, dk and dv in {16, 32}): whole and partial chunks, one token
    (2, 95, 2, 32, 32, "f32", "lm"),
    (1, 64, 3, 32, 16, "f32", "c0"),
    (2, 33, 1, 16, 32, "f32", "lm"),
    (1, 1, 2, 32, 32, "f32", "c0"),
]


@pytest.mark.parametrize("B,T,H,dk,dv,dtype,dist", SMALL)
@pytest.mark.parametrize("init", [False, True])
def test_forward_small(kla, B, T, H, dk, dv, dtype, dist, init):
    case = K.random_case(B, T, H, dk, dv, dtype, seed=T * 7 + dk, dist=dist)
    lam0, eta0 = _random_belief(B, H, dk, dv, T) if init else (None, None)
    log(f"forward small B{B} T{T} H{H} dk{dk} dv{dv} {dtype} init={init}")
    x = _dev_inputs(case, dtype)
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"],
                          None if lam0 is None else torch.tensor(lam0, dtype=torch.float32, device=DEV),
                          None if eta0 is None else torch.tensor(eta0, dtype=torch.float32, device=DEV),
                          want_var=True)
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0)
    rep = []
    _check("y", to_np(out["y"]), K.quantise(ref["y"], dtype) if dtype == "bf16" else ref["y"], TOL[dtype], rep)
    _check("yvar", to_np(out["yvar"]), ref["yvar"], TOL["f32"], rep)
    _check("lamT", to_np(out["lamT"]), ref["lamT"], TOL["f32"], rep)
    _check("etaT", to_np(out["etaT"]), ref["etaT"], TOL[dtype] if dtype == "bf16" else TOL["f32"], rep)
    assert np.all(to_np(out["lamT"]) > 0) and np.all(to_np(out["yvar"]) > 0)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("B,T,H,dk,dv,dtype,dist", SMALL)
@pytest.mark.parametrize("with_saved", [False, True])
def test_backward_small(kla, B, T, H, dk, dv, dtype, dist, with_saved):
    case = K.random_case(B, T, H, dk, dv, dtype, seed=T * 11 + dv, dist=dist)
    lam0, eta0 = _random_belief(B, H, dk, dv, T + 1)
    g = np.random.default_rng(T)
    dlamT = g.standard_normal((B, H, dk)).astype(np.float32).astype(np.float64)
    detaT = g.standard_normal((B, H, dk, dv)).astype(np.float32).astype(np.float64)
    dyvar = g.standard_normal((B, T, H)).astype(np.float32).astype(np.float64)
    log(f"backward small B{B} T{T} H{H} dk{dk} dv{dv} {dtype} saved={with_saved}")
    x = _dev_inputs(case, dtype)
    f32 = lambda a: torch.tensor(a, dtype=torch.float32, device=DEV)
    saved = None
    if with_saved:   # the context a forward with the same inputs saved
        saved = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0),
                                save=True)["saved"]
    gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), x["dy"],
                          f32(dlamT), f32(detaT), saved=saved, dyvar=f32(dyvar))
    torch.cuda.synchronize()
    ref = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0,
                          case["dy"], dlamT, detaT, dyvar=dyvar)
    rep = []
    for n in ("dq", "dk", "dv", "da", "dp", "dr"):
        _check(n, to_np(gr[n]), ref[n], TOL[dtype], rep)
    _check("dlam0", to_np(gr["dlam0"]), ref["dlam0"], TOL[dtype], rep)
    _check("deta0", to_np(gr["deta0"]), ref["deta0"], TOL[dtype], rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("dk,dv", [(32, 32), (128, 16)])
def test_backward_default_belief_ragged(kla, dk, dv):
    """fp32 paths (dk = dv = 32: the chunked fp64 one; dk = 128: the token-recurrent one)
    without an initial belief, final-belief gradients or a variance gradient, at a length
    that leaves a partial chunk or block."""
    B, T, H = 2, 37, 3
    case = K.random_case(B, T, H, dk, dv, "f32", seed=dk + dv, dist="c0")
    log(f"backward defaults B{B} T{T} H{H} dk{dk} dv{dv} f32")
    x = _dev_inputs(case, "f32")
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True)
    gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"])
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"])
    rg = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], None, None, case["dy"])
    rep = []
    _check("y", to_np(out["y"]), ref["y"], TOL["f32"], rep)
    _check("yvar", to_np(out["yvar"]), ref["yvar"], TOL["f32"], rep)
    for n in ("dq", "dk", "dv", "da", "dp", "dr"):
        _check(n, to_np(gr[n]), rg[n], TOL["f32"], rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("T", [15, 16, 31, 32, 33, 64, 65])
@pytest.mark.parametrize("dk,dv", [(32, 32), (64, 32)])
def test_recurrent_block_boundaries(kla, T, dk, dv):
    """The fp32 paths around their boundaries: the chunked fp64 path at dk = dv = 32
    (32-token chunks) and the token-recurrent path at dk = 64 (blocks of 16 / 32 tokens,
    state checkpoints every 64): forward with a saved context, backward from it and from
    a recomputed one (bitwise equal), against the oracle."""
    B, H = 2, 3
    case = K.random_case(B, T, H, dk, dv, "f32", seed=T + 101, dist="c0")
    lam0, eta0 = _random_belief(B, H, dk, dv, T + 7)
    g = np.random.default_rng(T + 5)
    dlamT = g.standard_normal((B, H, dk)).astype(np.float32).astype(np.float64)
    detaT = g.standard_normal((B, H, dk, dv)).astype(np.float32).astype(np.float64)
    log(f"recurrent boundaries B{B} T{T} H{H} dk{dk} dv{dv} f32")
    x = _dev_inputs(case, "f32")
    f32 = lambda a: torch.tensor(a, dtype=torch.float32, device=DEV)
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), want_var=True,
                          save=True)
    gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), x["dy"],
                          f32(dlamT), f32(detaT), saved=out["saved"])
    gr2 = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), x["dy"],
                           f32(dlamT), f32(detaT))
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0)
    rg = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0, case["dy"],
                         dlamT, detaT)
    rep = []
    for n in ("y", "yvar", "lamT", "etaT"):
        _check(n, to_np(out[n]), ref[n], TOL["f32"], rep)
    for n in ("dq", "dk", "dv", "da", "dp", "dr", "dlam0", "deta0"):
        _check(n, to_np(gr[n]), rg[n], TOL["f32"], rep)
        assert torch.equal(gr[n], gr2[n]), f"{n} differs between saved and recomputed context"
    log("  " + " ".join(rep))


@pytest.mark.parametrize("dk", [32, 64])   # fp32: the chunked fp64 path, the token-recurrent one
def test_empty_and_single_token(kla, dk):
    for T in (0, 1):
        case = K.random_case(2, T, 2, dk, 16, "f32", seed=5)
        lam0, eta0 = _random_belief(2, 2, dk, 16, 3)
        log(f"edge T={T} dk={dk}")
        x = _dev_inputs(case, "f32")
        f32 = lambda a: torch.tensor(a, dtype=torch.float32, device=DEV)
        out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), want_var=True)
        gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), x["dy"],
                              f32(np.ones((2, 2, dk))), f32(np.ones((2, 2, dk, 16))))
        torch.cuda.synchronize()
        ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0)
        rg = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0,
                             case["dy"], np.ones((2, 2, dk)), np.ones((2, 2, dk, 16)))
        np.testing.assert_allclose(to_np(out["lamT"]), ref["lamT"], rtol=1e-6)
        np.testing.assert_allclose(to_np(out["etaT"]), ref["etaT"], rtol=1e-6, atol=1e-7)
        np.testing.assert_allclose(to_np(gr["dlam0"]), rg["dlam0"], rtol=1e-5, atol=1e-6)
        np.testing.assert_allclose(to_np(gr["deta0"]), rg["deta0"], rtol=1e-5, atol=1e-6)
        if T:
            np.testing.assert_allclose(to_np(out["y"]), ref["y"], rtol=1e-5, atol=1e-6)


@pytest.mark.parametrize("T", [0, 1, 32, 33])
def test_chunked_edges(kla, T):
    """The chunked bf16 path with no token, one token, exactly one chunk and one chunk plus a token,
    with an initial belief and gradients of the final belief."""
    B, H, dk, dv = 2, 2, 64, 32
    case = K.random_case(B, T, H, dk, dv, "bf16", seed=50 + T, dist="lm")
    lam0, eta0 = _random_belief(B, H, dk, dv, 9)
    g = np.random.default_rng(T)
    dlamT = g.standard_normal((B, H, dk)).astype(np.float32).astype(np.float64)
    detaT = g.standard_normal((B, H, dk, dv)).astype(np.float32).astype(np.float64)
    log(f"chunked edge T={T}")
    x = _dev_inputs(case, "bf16")
    f32 = lambda a: torch.tensor(a, dtype=torch.float32, device=DEV)
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), want_var=True,
                          save=True)
    gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), x["dy"],
                          f32(dlamT), f32(detaT), saved=out["saved"])
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0)
    rg = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0,
                         case["dy"], dlamT, detaT)
    rep = []
    tol = TOL["bf16"]
    _check("lamT", to_np(out["lamT"]), ref["lamT"], TOL["f32"], rep)
    _check("etaT", to_np(out["etaT"]), ref["etaT"], tol, rep)
    _check("dlam0", to_np(gr["dlam0"]), rg["dlam0"], tol, rep)
    _check("deta0", to_np(gr["deta0"]), rg["deta0"], tol, rep)
    if T:
        _check("y", to_np(out["y"]), K.quantise(ref["y"], "bf16"), tol, rep)
        for n in ("dq", "dk", "dv", "da", "dp", "dr"):
            _check(n, to_np(gr[n]), rg[n], tol, rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("init", [False, True])
def test_segment_parallel_forward(kla, init):
    """Few long sequences take the segment-parallel forward (no saved context); it must agree with
    the oracle and with the one-pass chunked forward (taken when a saved context is asked for)."""
    B, T, H, dk, dv = 1, 8192, 2, 64, 64
    case = K.random_case(B, T, H, dk, dv, "bf16", seed=77, dist="lm")
    lam0, eta0 = _random_belief(B, H, dk, dv, 78) if init else (None, None)
    log(f"segment-parallel forward B{B} T{T} H{H} d{dk} init={init}")
    x = _dev_inputs(case, "bf16")
    f32 = lambda a: None if a is None else torch.tensor(a, dtype=torch.float32, device=DEV)
    seg = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), want_var=True)
    one = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], f32(lam0), f32(eta0), want_var=True,
                          save=True)
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0)
    rep = []
    tol = TOL["bf16"]
    for name, out in (("seg", seg), ("one", one)):
        _check(f"{name}.y", to_np(out["y"]), K.quantise(ref["y"], "bf16"), tol, rep)
        _check(f"{name}.yvar", to_np(out["yvar"]), ref["yvar"], TOL["f32"], rep)
        _check(f"{name}.lamT", to_np(out["lamT"]), ref["lamT"], TOL["f32"], rep)
        _check(f"{name}.etaT", to_np(out["etaT"]), ref["etaT"], tol, rep)
    log("  " + " ".join(rep))


def test_bitwise_deterministic(kla):
    case = K.random_case(2, 300, 4, 128, 128, "bf16", seed=9, dist="lm")
    x = _dev_inputs(case, "bf16")
    log("determinism")
    o1 = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True)
    o2 = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True)
    g1 = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"])
    g2 = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"])
    torch.cuda.synchronize()
    for a_, b_ in ((o1["y"], o2["y"]), (o1["etaT"], o2["etaT"]), (o1["yvar"], o2["yvar"])):
        assert torch.equal(a_, b_)
    for n in ("dq", "dk", "dv", "da", "dp", "dr", "dlam0", "deta0"):
        assert torch.equal(g1[n], g2[n]), n


def test_check_mode_rejects_out_of_domain(kla, monkeypatch):
    case = K.random_case(1, 40, 2, 16, 16, "f32", seed=3)
    case["a"][0, 5, 1, 3] = 1.5
    x = _dev_inputs(case, "f32")
    log("check mode")
    monkeypatch.setenv("KLA_CHECK", "1")
    with pytest.raises(kla.KLAError) as ei:
        kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"])
    assert ei.value.status == 6
    case["a"][0, 5, 1, 3] = 0.5
    x = _dev_inputs(case, "f32")
    kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"])   # valid input passes
    torch.cuda.synchronize()


def test_decode_steps_equal_forward(kla):
    B, T, H, dk, dv = 3, 20, 2, 64, 32
    case = K.random_case(B, T, H, dk, dv, "f32", seed=21, dist="lm")
    x = _dev_inputs(case, "f32")
    log("decode vs forward")
    full = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True)
    lam = torch.ones(B, H, dk, device=DEV)
    eta = torch.zeros(B, H, dk, dv, device=DEV)
    for t in range(T):
        sl = {n: x[n][:, t].contiguous() for n in K.NAMES}
        st = kla.kla_decode_step(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], lam, eta, want_var=True)
        torch.testing.assert_close(st["y"], full["y"][:, t], rtol=1e-5, atol=1e-6)
        torch.testing.assert_close(st["yvar"], full["yvar"][:, t], rtol=1e-5, atol=1e-6)
    torch.testing.assert_close(lam, full["lamT"], rtol=1e-5, atol=1e-6)
    torch.testing.assert_close(eta, full["etaT"], rtol=1e-5, atol=1e-6)


def test_autograd_wrapper(kla):
    case = K.random_case(1, 50, 2, 32, 32, "f32", seed=2)
    x = {n: to_torch(case[n], "f32", DEV).requires_grad_(True) for n in K.NAMES}
    log("autograd")
    y, yvar, lamT, etaT = kla.kla_filter(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True)
    dy = to_torch(case["dy"], "f32", DEV)
    gv = np.random.default_rng(3).standard_normal((1, 50, 2)).astype(np.float32).astype(np.float64)
    ((y * dy).sum() + (yvar * to_torch(gv, "f32", DEV)).sum()).backward()
    ref = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], None, None, case["dy"],
                          dyvar=gv)
    for n, gn in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("a", "da"), ("p", "dp"), ("r", "dr")):
        assert rel_err(to_np(x[n].grad), ref[gn]) <= TOL["f32"], n


# ------------------------------------------------------------------ workloads
def _sample_pairs(w, count, seed=0):
    g = np.random.default_rng(seed)
    pairs = {(0, 0), (w.B - 1, w.H - 1)}
    while len(pairs) < min(count, w.B * w.H):
        pairs.add((int(g.integers(w.B)), int(g.integers(w.H))))
    return sorted(pairs)


def _workload_parity(kla, cid, pairs_n, backward):
    w = K.WORKLOADS[cid]
    log(f"workload {cid} ({w.name}) B{w.B} T{w.T} H{w.H} d{w.dk} {w.dtype}: generating inputs")
    bits = K.full(w, as_bits=True)
    x = {n: bits_to_torch(bits[n], DEV) for n in bits}
    del bits
    log(f"workload {cid}: forward on GPU")
    # the launch configuration bench.py times: the forward saves its context for the backward
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True, save=backward)
    gr = None
    if backward:
        log(f"workload {cid}: backward on GPU")
        gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"],
                              saved=out["saved"])
    torch.cuda.synchronize()
    pairs = _sample_pairs(w, pairs_n)
    log(f"workload {cid}: oracle on pairs {pairs}")
    sl = K.pairs_slice(w, pairs)
    ref = oracle.forward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"])
    rg = oracle.backward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], None, None, sl["dy"]) \
        if backward else None
    tol = TOL[w.dtype]
    rep = []
    bi = [b for b, _ in pairs]
    hi = [h for _, h in pairs]
    got_y = to_np(out["y"][bi, :, hi])            # [n, T, dv]
    ref_y = ref["y"][:, :, 0]
    _check("y", got_y, K.quantise(ref_y, w.dtype), tol, rep)
    _check("yvar", to_np(out["yvar"][bi, :, hi]), ref["yvar"][:, :, 0], TOL["f32"] if w.dtype == "f32" else tol, rep)
    _check("lamT", to_np(out["lamT"][bi, hi]), ref["lamT"][:, 0], TOL["f32"] if w.dtype == "f32" else tol, rep)
    _check("etaT", to_np(out["etaT"][bi, hi]), ref["etaT"][:, 0], tol, rep)
    assert torch.all(out["lamT"] > 0) and torch.all(out["yvar"] > 0)
    assert torch.isfinite(out["y"].float()).all()
    if backward:
        for n in ("dq", "dk", "dv", "da", "dp", "dr"):
            _check(n, to_np(gr[n][bi, :, hi]), rg[n][:, :, 0], tol, rep)
        for n in ("dq", "dk", "dv", "da", "dp", "dr"):
            assert torch.isfinite(gr[n].float()).all(), n
    log(f"  workload {cid}: " + " ".join(rep))


def test_workload0_tiny_forward(kla):
    _workload_parity(kla, 0, 2, backward=True)


def test_workload1_state_tracking_fwd_bwd(kla):
    _workload_parity(kla, 1, 32, backward=True)


def test_workload2_lm_layer_fwd_bwd(kla):
    _workload_parity(kla, 2, 12, backward=True)


def test_workload3_long_context_forward(kla):
    w = K.WORKLOADS[3]
    # the corner pairs (heads 0 and 15: a normal-gate head and a near-one-gate head) and six more
    _workload_parity(kla, 3, 8, backward=False)


def test_workload4_decode(kla):
    w = K.WORKLOADS[4]
    S, H, d = w.B, w.H, w.dk
    log(f"workload 4: prewarm inputs S{S} T{w.T} H{H} d{d}")
    bits = K.full(w, names=K.NAMES, as_bits=True)
    x = {n: bits_to_torch(bits[n], DEV) for n in bits}
    del bits
    pre = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"])
    del x
    lam, eta = pre["lamT"], pre["etaT"]
    log("workload 4: decode inputs")
    steps = w.extra["steps"]
    dbits = K.decode_inputs(w, as_bits=True)
    dx = {n: bits_to_torch(dbits[n], DEV) for n in dbits}
    del dbits
    pairs = _sample_pairs(w, 8)
    bi = [b for b, _ in pairs]
    hi = [h for _, h in pairs]
    ys = []
    log("workload 4: 256 decode steps")
    for t in range(steps):
        sl = {n: dx[n][:, t].contiguous() for n in K.NAMES}
        st = kla.kla_decode_step(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], lam, eta)
        ys.append(st["y"][bi, hi].clone())
    torch.cuda.synchronize()
    log(f"workload 4: oracle on pairs {pairs} (1280-token sequential filter)")
    pre_sl = K.pairs_slice(w, pairs, names=K.NAMES)
    w2 = K.Workload(w.cid, w.name, w.B, steps, w.H, w.dk, w.dv, w.dtype, w.dist, False)
    dec_sl = K.pairs_slice(w2, pairs, names=K.NAMES, seed=w.cid + 1000)
    cat = {n: np.concatenate([pre_sl[n], dec_sl[n]], axis=1) for n in K.NAMES}
    ref = oracle.forward(cat["q"], cat["k"], cat["v"], cat["a"], cat["p"], cat["r"])
    rep = []
    got_y = np.stack([to_np(y) for y in ys], axis=1)      # [n, steps, dv]
    _check("y_decode", got_y, ref["y"][:, w.T:, 0], TOL["f32"], rep)
    _check("lam", to_np(lam[bi, hi]), ref["lamT"][:, 0], TOL["f32"], rep)
    _check("eta", to_np(eta[bi, hi]), ref["etaT"][:, 0], TOL["f32"], rep)
    assert torch.all(lam > 0)
    log("  workload 4: " + " ".join(rep))
