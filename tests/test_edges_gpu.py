"""GPU edge cases of the filter path, each against a reference that does not come from
the GPU: the zero-process-noise closed form, the oracle at boundary gate values, the
oracle's own belief for a decode continuation, and the range guard of the chunked walk.

* pbar = 0 with a time-invariant abar per key slot: lam and the state have closed forms
  (the appendix theorem with the initial-belief terms and sums from s = 1, reading R8),
  on the chunked path (bf16) and the chunked fp64 path (fp32, dk = 32, dv = 16).
* abar = 1 exactly, and small abar with tiny pbar (the gate F = abar rho then exceeds 1
  for the first tokens), against the oracle on the three paths (bf16 chunked, fp32
  token-recurrent at dk = 64, fp32 chunked fp64 at dk = dv = 32).
* Split-sequence resume: two forwards chained through the final belief equal one
  forward over the whole sequence; the cut at token 45 is not a multiple of the 32-token
  chunk, so the chunk boundaries of the second part move by 13 tokens (the results do
  not depend on where chunks start).
* Decode seeded with the oracle's belief after a 1024-token prewarm, compared step by
  step with the oracle's continuation.
* KLA_CHECK=1 reports KLA_ERR_RANGE when the gate products of a chunk leave the walk's
  range (bf16 inputs: abar = 0.03 over whole chunks underflows fp32; fp32 inputs:
  abar = 1e-12 underflows fp64), and passes in range.
"""
import numpy as np
import pytest

import kla_inputs as K
import oracle
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


def _dev(case, dtype, names=K.NAMES):
    return {n: to_torch(case[n], dtype, DEV) for n in names}


def _closed_form_pbar0(q, k, v, abar, r, lam0, eta0):
    """pbar = 0, abar[b, h, n] the same for every token: lam_t = abar^-2t lam0 +
    sum_{s<=t} abar^-2(t-s) k_s^2 r_s and H_t = abar^-t eta0 + sum_{s<=t} abar^-(t-s)
    r_s k_s v_s, in fp64 from the inputs alone."""
    B, T, H, dk = q.shape
    t = np.arange(1, T + 1, dtype=np.float64)
    y = np.empty(v.shape)
    lamT = np.empty((B, H, dk))
    etaT = np.empty((B, H, dk, v.shape[-1]))
    for b in range(B):
        for h in range(H):
            a = abar[b, h]                                    # [dk]
            w2 = a[None, :] ** (-2.0 * t[:, None])            # abar^-2t  [T, dk]
            w1 = a[None, :] ** (-1.0 * t[:, None])            # abar^-t
            kr = k[b, :, h] * r[b, :, h, None]                # r_s k_s  [T, dk]
            lam = w2 * (lam0[b, h][None, :] + np.cumsum(k[b, :, h] * kr / w2, axis=0))
            Hs = w1[:, :, None] * (eta0[b, h][None] + np.cumsum((kr / w1)[:, :, None] * v[b, :, h][:, None, :],
                                                                axis=0))
            y[b, :, h] = np.einsum("tn,tnd->td", q[b, :, h] / lam, Hs)
            lamT[b, h], etaT[b, h] = lam[-1], Hs[-1]
    return {"y": y, "lamT": lamT, "etaT": etaT}


@pytest.mark.parametrize("dtype,dk,dv", [("bf16", 64, 32), ("f32", 32, 16)])
def test_zero_process_noise_closed_form(kla, dtype, dk, dv):
    B, T, H = 2, 70, 2
    case = K.random_case(B, T, H, dk, dv, dtype, seed=81, dist="lm")
    g = np.random.default_rng(82)
    abar = K.quantise(0.9 + 0.1 * g.random((B, H, dk)), dtype)
    case["a"] = np.broadcast_to(abar[:, None], (B, T, H, dk)).copy()
    case["p"] = np.zeros((B, T, H, dk))
    lam0 = K.quantise(0.5 + g.random((B, H, dk)), "f32")
    eta0 = K.quantise(g.standard_normal((B, H, dk, dv)), "f32")
    log(f"pbar = 0 closed form {dtype} dk{dk} dv{dv}")
    x = _dev(case, dtype)
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], to_torch(lam0, "f32", DEV),
                          to_torch(eta0, "f32", DEV), want_state=True)
    torch.cuda.synchronize()
    ref = _closed_form_pbar0(case["q"], case["k"], case["v"], abar, case["r"], lam0, eta0)
    orc = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], lam0, eta0)
    rep = []
    for n in ("y", "lamT", "etaT"):
        _check(n, to_np(out[n]), ref[n], TOL[dtype], rep)
        np.testing.assert_allclose(orc[n], ref[n], rtol=1e-9, atol=1e-9 * np.abs(ref[n]).max())
    log("  " + " ".join(rep))


def _gates(kind, B, T, H, dk, g):
    if kind == "abar_one":
        return np.ones((B, T, H, dk)), 0.05 * g.random((B, T, H, dk))
    # small abar, tiny pbar: F = abar rho is about 1 / abar until p lam reaches abar^2
    return 0.25 + 0.1 * g.random((B, T, H, dk)), 1e-4 * g.random((B, T, H, dk))


@pytest.mark.parametrize("kind", ["abar_one", "small_abar_tiny_pbar"])
@pytest.mark.parametrize("dtype,dk,dv", [("bf16", 128, 64), ("f32", 64, 32), ("f32", 32, 32)])
def test_boundary_gates_against_oracle(kla, kind, dtype, dk, dv):
    B, T, H = 2, 75, 2
    case = K.random_case(B, T, H, dk, dv, dtype, seed=91, dist="lm")
    g = np.random.default_rng(92)
    a, p = _gates(kind, B, T, H, dk, g)
    case["a"], case["p"] = K.quantise(a, dtype), K.quantise(p, dtype)
    dlamT = K.quantise(g.standard_normal((B, H, dk)), "f32")
    log(f"boundary gates {kind} {dtype} dk{dk} dv{dv}")
    x = _dev(case, dtype, K.NAMES + ("dy",))
    out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_state=True, want_var=True)
    gr = kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"],
                          to_torch(dlamT, "f32", DEV))
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"])
    rg = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], None, None, case["dy"],
                         dlamT)
    rep = []
    for n in ("y", "yvar", "lamT", "etaT"):
        _check(n, to_np(out[n]), ref[n], TOL[dtype], rep)
    for n in ("dq", "dk", "dv", "da", "dp", "dr"):
        _check(n, to_np(gr[n]), rg[n], TOL[dtype], rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("dtype,dk,dv", [("bf16", 128, 128), ("f32", 64, 32), ("f32", 32, 32)])
def test_split_sequence_resume(kla, dtype, dk, dv):
    B, T, H, cut = 2, 100, 2, 45
    case = K.random_case(B, T, H, dk, dv, dtype, seed=101, dist="lm")
    log(f"split-sequence resume {dtype} dk{dk} dv{dv} cut {cut}")
    x = _dev(case, dtype)
    first = {n: t[:, :cut].contiguous() for n, t in x.items()}
    second = {n: t[:, cut:].contiguous() for n, t in x.items()}
    whole = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_state=True)
    p1 = kla.kla_forward(first["q"], first["k"], first["v"], first["a"], first["p"], first["r"], want_state=True)
    p2 = kla.kla_forward(second["q"], second["k"], second["v"], second["a"], second["p"], second["r"],
                         p1["lamT"], p1["etaT"], want_state=True)
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"])
    rep = []
    _check("y_first", to_np(p1["y"]), ref["y"][:, :cut], TOL[dtype], rep)
    _check("y_second", to_np(p2["y"]), ref["y"][:, cut:], TOL[dtype], rep)
    _check("y_second_vs_whole", to_np(p2["y"]), to_np(whole["y"])[:, cut:], TOL[dtype], rep)
    _check("lamT", to_np(p2["lamT"]), ref["lamT"], TOL[dtype], rep)
    _check("etaT", to_np(p2["etaT"]), ref["etaT"], TOL[dtype], rep)
    _check("etaT_vs_whole", to_np(p2["etaT"]), to_np(whole["etaT"]), TOL[dtype], rep)
    log("  " + " ".join(rep))


def test_decode_from_oracle_belief(kla):
    """Decode seeded with the oracle's belief after a 1024-token prewarm (the decode
    workload's distributions at S = 8 sequences), 64 steps against the oracle."""
    S, H, d, T0, steps = 8, 4, 128, 1024, 64
    w = K.Workload(-1, "decode_small", S, T0, H, d, d, "f32", "lm", True)
    pre = K.full(w, names=K.NAMES, seed=41)
    w2 = K.Workload(-1, "decode_small", S, steps, H, d, d, "f32", "lm", True)
    dec = K.full(w2, names=K.NAMES, seed=41 + 1000)
    log("decode from the oracle's belief: oracle prewarm")
    warm = oracle.forward(pre["q"], pre["k"], pre["v"], pre["a"], pre["p"], pre["r"])
    lam0 = K.quantise(warm["lamT"], "f32")
    eta0 = K.quantise(warm["etaT"], "f32")
    ref = oracle.forward(dec["q"], dec["k"], dec["v"], dec["a"], dec["p"], dec["r"], lam0, eta0)
    lam = to_torch(lam0, "f32", DEV)
    eta = to_torch(eta0, "f32", DEV)
    x = _dev(dec, "f32")
    ys, yvs = [], []
    log("decode from the oracle's belief: 64 steps")
    for t in range(steps):
        sl = {n: x[n][:, t].contiguous() for n in K.NAMES}
        st = kla.kla_decode_step(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], lam, eta, want_var=True)
        ys.append(to_np(st["y"]))
        yvs.append(to_np(st["yvar"]))
    torch.cuda.synchronize()
    rep = []
    got = np.stack(ys, axis=1)
    for t in (0, 1, steps // 2, steps - 1):   # step by step, then the whole run
        _check(f"y_step{t}", got[:, t], ref["y"][:, t], TOL["f32"], rep)
    _check("y", got, ref["y"], TOL["f32"], rep)
    _check("yvar", np.stack(yvs, axis=1), ref["yvar"], TOL["f32"], rep)
    _check("lam", to_np(lam), ref["lamT"], TOL["f32"], rep)
    _check("eta", to_np(eta), ref["etaT"], TOL["f32"], rep)
    log("  " + " ".join(rep))


# abar whose product over a 32-token chunk leaves the walk's range: fp32 arithmetic for bf16
# inputs (0.03^32 ~ 2e-49), fp64 for fp32 inputs (1e-12 per token leaves fp64 after 26 tokens)
@pytest.mark.parametrize("dtype,dk,dv,abar", [("bf16", 64, 32, 0.03), ("f32", 32, 32, 1e-12)])
def test_chunk_range_guard(kla, monkeypatch, dtype, dk, dv, abar):
    B, T, H = 1, 96, 2
    case = K.random_case(B, T, H, dk, dv, dtype, seed=111, dist="lm")
    good = _dev(case, dtype, K.NAMES + ("dy",))
    bad_case = dict(case)
    bad_case["a"] = K.quantise(np.full((B, T, H, dk), abar), dtype)
    bad_case["p"] = K.quantise(np.full((B, T, H, dk), 0.05), dtype)
    bad = _dev(bad_case, dtype, K.NAMES + ("dy",))
    log(f"chunk range guard {dtype} dk{dk} dv{dv} abar={abar}")
    monkeypatch.setenv("KLA_CHECK", "1")
    with pytest.raises(kla.KLAError) as ei:
        kla.kla_forward(bad["q"], bad["k"], bad["v"], bad["a"], bad["p"], bad["r"])
    assert ei.value.status == 8
    with pytest.raises(kla.KLAError) as ei:
        kla.kla_backward(bad["q"], bad["k"], bad["v"], bad["a"], bad["p"], bad["r"], None, None, bad["dy"])
    assert ei.value.status == 8
    # inside the range both calls pass, and the flag of the failed calls does not linger
    out = kla.kla_forward(good["q"], good["k"], good["v"], good["a"], good["p"], good["r"], save=True)
    kla.kla_backward(good["q"], good["k"], good["v"], good["a"], good["p"], good["r"], None, None, good["dy"],
                     saved=out["saved"])
    torch.cuda.synchronize()
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"])
    assert rel_err(to_np(out["y"]), ref["y"]) <= TOL[dtype]
