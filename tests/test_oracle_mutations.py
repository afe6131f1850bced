"""Planted mistakes: each mutation of a copy of the oracle's C source must be caught.

A mistake is planted in a temporary copy of ``oracle/kla_oracle.c`` (never in
the real one), compiled on the CPU, and run through a compact battery made of
two independent pins -- the covariance-form Kalman filter and central finite
differences -- which must then fail.  This shows the pins can see a dropped
term, a wrong sign, a wrong index or a wrong factor anywhere in the oracle.
"""
import importlib.util
import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "kla_oracle.c")

MUTATIONS = {
    "drop_process_noise": ("1.0 / (an * an + pn * (*L));", "1.0 / (an * an + 0.0 * (*L));"),
    "forget_gate_without_decay": ("double f = an * rho;", "double f = rho;"),
    "precision_wrong_channel": ("*L = rho * (*L) + kt[n] * kt[n] * rt[d];", "*L = rho * (*L) + kt[n] * kt[n] * rt[0];"),
    "evidence_missing_key": ("*E = f * (*E) + kt[n] * rt[d] * vt[d];", "*E = f * (*E) + rt[d] * vt[d];"),
    "readout_without_precision": ("yt[d] += qt[n] * (*E) * inv;", "yt[d] += qt[n] * (*E);"),
    "variance_query_not_squared": ("wt[d] += qt[n] * qt[n] * inv;", "wt[d] += qt[n] * inv;"),
    "bwd_mean_adjoint_sign": ("gl -= dmu * ec / (lc * lc);", "gl += dmu * ec / (lc * lc);"),
    "bwd_noise_grad_wrong_index": ("double dpt = dden * lp;", "double dpt = dden * lc;"),
    "bwd_key_grad_missing_factor": ("J->dk_[ik] += gl * 2.0 * k * r;", "J->dk_[ik] += gl * k * r;"),
    "bwd_gate_adjoint_dropped": ("gl_prev += dden * p;", "gl_prev += 0.0;"),
    "bwd_variance_query_factor": ("J->dq[ik] += 2.0 * q * gv / lc;", "J->dq[ik] += q * gv / lc;"),
    "bwd_variance_precision_power": ("gl -= q * q * gv / (lc * lc);", "gl -= q * q * gv / lc;"),
    # gates per (key slot, value channel)
    "nd_gate_transposed": ("if (J->gate_nd) return ((size_t)h * J->dk + n) * J->dv + d;",
                           "if (J->gate_nd) return ((size_t)h * J->dv + d) * J->dk + n;"),
    "nd_gate_of_slot_only": ("if (J->gate_nd) return ((size_t)h * J->dk + n) * J->dv + d;",
                             "if (J->gate_nd) return ((size_t)h * J->dk + n) * J->dv;"),
    "nd_gate_grad_sum_dropped": ("            sa += dat;\n", "            sa += 0.0 * dat;\n"),
}


def _load_mutant(tmp_path, name):
    src = open(SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, f"mutation anchor not unique/present: {old}"
    mut_dir = tmp_path / name
    mut_dir.mkdir()
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), mut_dir / "__init__.py")
    (mut_dir / "kla_oracle.c").write_text(src.replace(old, new))
    lib = mut_dir / "_kla_oracle.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-ffp-contract=off",
                    str(mut_dir / "kla_oracle.c"), "-o", str(lib), "-lm"], check=True)
    spec = importlib.util.spec_from_file_location(f"oracle_{name}", mut_dir / "__init__.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert mod._LIB_PATH == str(lib)
    return mod


def _kf_battery(orc) -> bool:
    """True when the oracle agrees with the textbook covariance-form filter."""
    g = np.random.default_rng(0)
    T, dk, dv = 12, 3, 2
    q, k = g.standard_normal((2, 1, T, 1, dk))
    v = g.standard_normal((1, T, 1, dv))
    a = 0.5 + 0.5 * g.random((1, T, 1, dk))
    p = 0.1 + g.random((1, T, 1, dk))
    r = 0.2 + g.random((1, T, 1, dv))
    out = orc.forward(q, k, v, a, p, r)
    Sig = np.ones((dk, dv))
    mu = np.zeros((dk, dv))
    ok = True
    for t in range(T):
        at, pt, kt = a[0, t, 0][:, None], p[0, t, 0][:, None], k[0, t, 0][:, None]
        rt, vt = r[0, t, 0][None, :], v[0, t, 0][None, :]
        mp = at * mu
        Sp = at * at * Sig + pt
        K = Sp * kt / (kt * kt * Sp + 1.0 / rt)
        mu = mp + K * (vt - kt * mp)
        Sig = (1.0 - K * kt) * Sp
        ok &= np.allclose(out["y"][0, t, 0], (q[0, t, 0][:, None] * mu).sum(0), rtol=1e-9, atol=1e-12)
        ok &= np.allclose(out["yvar"][0, t, 0], (q[0, t, 0][:, None] ** 2 * Sig).sum(0), rtol=1e-9)
    ok &= np.allclose(out["lamT"][0, 0], 1.0 / Sig, rtol=1e-9)
    return bool(ok)


def _fd_battery(orc) -> bool:
    """True when the oracle's gradient agrees with central differences of its forward."""
    g = np.random.default_rng(1)
    B, T, H, dk, dv = 1, 5, 1, 2, 2
    inp = dict(q=g.standard_normal((B, T, H, dk)), k=g.standard_normal((B, T, H, dk)),
               v=g.standard_normal((B, T, H, dv)), a=0.5 + 0.5 * g.random((B, T, H, dk)),
               p=0.1 + g.random((B, T, H, dk)), r=0.2 + g.random((B, T, H)),
               lam0=0.5 + g.random((B, H, dk)), eta0=g.standard_normal((B, H, dk, dv)))
    dy = g.standard_normal((B, T, H, dv))
    dlamT = g.standard_normal((B, H, dk))
    detaT = g.standard_normal((B, H, dk, dv))
    dyvar = g.standard_normal((B, T, H))

    def loss():
        o = orc.forward(inp["q"], inp["k"], inp["v"], inp["a"], inp["p"], inp["r"], inp["lam0"], inp["eta0"])
        return ((o["y"] * dy).sum() + (o["lamT"] * dlamT).sum() + (o["etaT"] * detaT).sum()
                + (o["yvar"] * dyvar).sum())

    gr = orc.backward(inp["q"], inp["k"], inp["v"], inp["a"], inp["p"], inp["r"], inp["lam0"], inp["eta0"],
                      dy, dlamT, detaT, dyvar=dyvar)
    ok = True
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("a", "da"), ("p", "dp"), ("r", "dr"),
                        ("lam0", "dlam0"), ("eta0", "deta0")):
        x = inp[name]
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + 1e-6
            lp = loss()
            x[idx] = old - 1e-6
            lm = loss()
            x[idx] = old
            fd[idx] = (lp - lm) / 2e-6
        ok &= np.allclose(gr[gname], fd, rtol=1e-5, atol=1e-6)
    return bool(ok)


def _nd_battery(orc) -> bool:
    """Gates per (n, d): the textbook covariance-form filter per element, and central
    differences of the gate gradients."""
    g = np.random.default_rng(2)
    B, T, H, dk, dv = 1, 7, 1, 3, 2
    q, k = g.standard_normal((2, B, T, H, dk))
    v = g.standard_normal((B, T, H, dv))
    r = 0.2 + g.random((B, T, H, dv))
    a = 0.3 + 0.6 * g.random((H, dk, dv))
    p = 0.05 + g.random((H, dk, dv))
    out = orc.forward_nd(q, k, v, a, p, r)
    Sig, mu, ok = np.ones((dk, dv)), np.zeros((dk, dv)), True
    for t in range(T):
        kt = k[0, t, 0][:, None]
        mp = a[0] * mu
        Sp = a[0] ** 2 * Sig + p[0]
        K = Sp * kt / (kt * kt * Sp + 1.0 / r[0, t, 0][None, :])
        mu = mp + K * (v[0, t, 0][None, :] - kt * mp)
        Sig = (1.0 - K * kt) * Sp
        ok &= np.allclose(out["y"][0, t, 0], (q[0, t, 0][:, None] * mu).sum(0), rtol=1e-9, atol=1e-12)
    dy = g.standard_normal((B, T, H, dv))
    gr = orc.backward_nd(q, k, v, a, p, r, None, None, dy)
    loss = lambda aa, pp: float((orc.forward_nd(q, k, v, aa, pp, r)["y"] * dy).sum())
    for x, gname in ((a, "g_abar"), (p, "g_pbar")):
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + 1e-6
            lp = loss(a, p)
            x[idx] = old - 1e-6
            lm = loss(a, p)
            x[idx] = old
            ok &= abs((lp - lm) / 2e-6 - gr[gname][idx]) < 1e-5 * max(1.0, abs(gr[gname][idx]))
    return bool(ok)


def test_unmutated_copy_passes_battery(tmp_path):
    import oracle
    assert _kf_battery(oracle) and _fd_battery(oracle) and _nd_battery(oracle)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    orc = _load_mutant(tmp_path, name)
    assert not (_kf_battery(orc) and _fd_battery(orc) and _nd_battery(orc)), f"mutation {name} went unnoticed"
