"""GPU parity of the Monte Carlo readout of KLA+ (kla_mc_sample, kla_mc_sample_backward,
kla_mc_nll, kla_mc_nll_backward) against the fp64 oracle (oracle/mc.py), element by
element, including the draws (both sides run Philox4x64-10 from the same counters),
and the whole KLA+ objective end to end: layer forward, draws, a linear decoder,
logsumexp over the draws, and every gradient back to the layer's inputs."""
import numpy as np
import pytest

import kla_inputs as K
import oracle
from oracle import mc
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
    report.append(f"{name}={e:.2e}(rms-rel {rel_err(got, ref, 1.0):.1e})")
    assert np.all(np.isfinite(got)), f"{name} has non-finite values"
    assert e <= tol, f"{name}: rel err {e:.3e} > {tol:.0e}"


CASES = [  # B, T, H, dv, dtype, S, seed
    (2, 37, 3, 16, "f32", 4, 1),
    (1, 64, 2, 128, "bf16", 10, 2),
    (1, 5, 1, 32, "f32", 1, 3),
    (3, 20, 2, 64, "bf16", 3, 2**64 - 5),
]


@pytest.mark.parametrize("B,T,H,dv,dtype,S,seed", CASES)
def test_mc_sample_and_backward(kla, B, T, H, dv, dtype, S, seed):
    g = np.random.default_rng(seed % 1000)
    ymu = K.quantise(g.standard_normal((B, T, H, dv)), dtype)
    yvar = K.quantise(0.05 + g.random((B, T, H)) * 2.0, "f32")
    dys = K.quantise(g.standard_normal((S, B, T, H, dv)), dtype)
    log(f"mc sample B{B} T{T} H{H} dv{dv} {dtype} S{S}")
    ys = kla.kla_mc_sample(to_torch(ymu, dtype, DEV), to_torch(yvar, "f32", DEV), S, seed)
    dymu, dyvar = kla.kla_mc_sample_backward(to_torch(yvar, "f32", DEV), to_torch(dys, dtype, DEV), seed)
    torch.cuda.synchronize()
    ref = mc.mc_sample(ymu, yvar, S, seed)
    rdymu, rdyvar = mc.mc_sample_backward(yvar, dys, seed)
    rep = []
    tol = TOL[dtype]
    _check("ys", to_np(ys), K.quantise(ref, dtype) if dtype == "bf16" else ref, tol, rep)
    _check("dymu", to_np(dymu), rdymu, tol, rep)
    _check("dyvar", to_np(dyvar), rdyvar, TOL["f32"] if dtype == "f32" else tol, rep)
    log("  " + " ".join(rep))


@pytest.mark.parametrize("S,n", [(1, 100), (10, 1000), (7, 4099)])
def test_mc_nll_and_backward(kla, S, n):
    g = np.random.default_rng(S + n)
    logp = K.quantise(-np.abs(g.standard_normal((S, n))) * 4.0, "f32")
    logp[:, :3] -= 200.0                     # far tails: the logsumexp form stays finite
    dnll = K.quantise(g.standard_normal(n), "f32")
    log(f"mc nll S{S} n{n}")
    lp = to_torch(logp, "f32", DEV)
    nll = kla.kla_mc_nll(lp)
    dlogp = kla.kla_mc_nll_backward(lp, to_torch(dnll, "f32", DEV))
    torch.cuda.synchronize()
    rep = []
    _check("nll", to_np(nll), mc.mc_nll(logp), TOL["f32"], rep)
    _check("dlogp", to_np(dlogp), mc.mc_nll_backward(logp, dnll), TOL["f32"], rep)
    log("  " + " ".join(rep))


def test_mc_sample_lm_shape_sampled_rows(kla):
    """The LM-layer shape (B8 T2048 H16 dv128, bf16) with S = 10 draws: every draw of a sample
    of rows against the oracle, which draws eps for exactly those flat indices."""
    B, T, H, dv, S, seed = 8, 2048, 16, 128, 10, 2026
    g = np.random.default_rng(0)
    ymu_bits = K.bf16_bits(g.standard_normal((B, T, H, dv)))
    yvar = K.quantise(0.05 + g.random((B, T, H)), "f32")
    log("mc sample LM shape: draws on the GPU")
    ymu_t = torch.from_numpy(ymu_bits.view(np.int16)).view(torch.bfloat16).to(DEV)
    ys = kla.kla_mc_sample(ymu_t, to_torch(yvar, "f32", DEV), S, seed)
    torch.cuda.synchronize()
    rows = np.array([0, 1, 12345, 262143, 99999, 200003])    # flat (b, t, h) rows
    nrow = B * T * H
    ymu_f = K.bf16_to_f64(ymu_bits).reshape(nrow, dv)
    got = to_np(ys.view(S, nrow, dv)[:, torch.as_tensor(rows, device=DEV)])
    e = (np.arange(S)[:, None, None] * nrow + rows[None, :, None]) * dv + np.arange(dv)[None, None, :]
    ref = ymu_f[rows][None] + np.sqrt(yvar.reshape(nrow)[rows])[None, :, None] * mc.normals(e, seed)
    rep = []
    _check("ys", got, K.quantise(ref, "bf16"), TOL["bf16"], rep)
    assert torch.isfinite(ys.float()).all()
    log("  " + " ".join(rep))


@pytest.mark.parametrize("dtype", ["f32"])
def test_kla_plus_objective_end_to_end(kla, dtype):
    """Layer forward (y, yvar), S draws, a linear decoder with log-softmax at target tokens,
    -logsumexp over the draws + log S, summed over tokens; the gradients of every layer
    input through the library's backward kernels against the same chain in fp64.

    fp32 only: in bf16 each stage's input is the previous stage's bf16 output, which differs
    from the rounded fp64 value by a bf16 ulp in some elements, and the decoder carries that
    into the upstream gradient of the backward; the bf16 stages are checked one by one (the
    draws and their backward above, the layer's backward in the filter's own parity tests)."""
    B, T, H, dk, dv, S, V, seed = 2, 40, 2, 32, 32, 5, 11, 77
    case = K.random_case(B, T, H, dk, dv, dtype, seed=5, dist="lm")
    g = np.random.default_rng(6)
    W = K.quantise(g.standard_normal((dv, V)) / np.sqrt(dv), "f32")
    tgt = g.integers(0, V, size=(B, T, H))
    log(f"KLA+ objective end to end {dtype}")
    x = {n: to_torch(case[n], dtype, DEV).requires_grad_(True) for n in K.NAMES}
    Wt = to_torch(W, "f32", DEV)
    tg = torch.as_tensor(tgt, device=DEV)

    def decoder_logp(ys):   # [S, B, T, H, dv] -> log p(target | draw) [S, B, T, H]
        lp = torch.log_softmax(ys.float() @ Wt, dim=-1)
        return torch.gather(lp, -1, tg.expand(ys.shape[0], -1, -1, -1).unsqueeze(-1)).squeeze(-1).contiguous()

    y, yvar, _, _ = kla.kla_filter(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_var=True)
    nll = kla.kla_mc_nll_loss(y, yvar, decoder_logp, S=S, seed=seed)
    nll.sum().backward()
    torch.cuda.synchronize()

    # the same chain in fp64: oracle forward, draws, decoder, loss, and back
    ref = oracle.forward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"])
    ys = mc.mc_sample(ref["y"], ref["yvar"], S, seed)
    logits = ys @ W
    lse = logits.max(-1, keepdims=True)
    lse = lse + np.log(np.exp(logits - lse).sum(-1, keepdims=True))
    logsm = logits - lse
    logp = np.take_along_axis(logsm, np.broadcast_to(tgt, (S,) + tgt.shape)[..., None], -1)[..., 0]
    nll_r = mc.mc_nll(logp.reshape(S, -1)).reshape(tgt.shape)
    dlogp = mc.mc_nll_backward(logp.reshape(S, -1), np.ones(tgt.size)).reshape(logp.shape)
    onehot = np.eye(V)[np.broadcast_to(tgt, (S,) + tgt.shape)]
    dlogits = dlogp[..., None] * (onehot - np.exp(logsm))
    dys = dlogits @ W.T
    dymu, dyvar = mc.mc_sample_backward(ref["yvar"], dys, seed)
    rg = oracle.backward(case["q"], case["k"], case["v"], case["a"], case["p"], case["r"], None, None, dymu,
                         dyvar=dyvar)
    rep = []
    tol = TOL[dtype]
    _check("nll", to_np(nll), nll_r, tol, rep)
    for n, gn in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("a", "da"), ("p", "dp"), ("r", "dr")):
        _check(gn, to_np(x[n].grad), rg[gn], tol, rep)
    log("  " + " ".join(rep))
