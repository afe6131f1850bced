"""Pins of the oracle with gates per (key slot, value channel) -- Algorithm 1's
Abar, Pbar : (N, D), time-invariant, with the observation precision per value
channel -- on the CPU.

* With gates that do not depend on the channel it equals the per-slot form (the
  oracle path pinned in test_oracle_pins.py) for every output and gradient.
* Every element (n, d) is the textbook covariance-form Kalman filter with its own
  gates (the KF column of the paper's KF/IF table), element by element.
* Central finite differences of every gradient, the per-(n, d) gates included, and
  of the OU parameters (Sec. 4.1's discretisation applied per element).
* The masses of the parameter-gradient sums bound the sums and equal them for a
  single term.
"""
import numpy as np
import pytest

import oracle


def _inputs(seed, B=2, T=9, H=2, dk=3, dv=4):
    g = np.random.default_rng(seed)
    return dict(q=g.standard_normal((B, T, H, dk)), k=g.standard_normal((B, T, H, dk)),
                v=g.standard_normal((B, T, H, dv)), r=0.2 + g.random((B, T, H, dv)),
                a=0.3 + 0.65 * g.random((H, dk, dv)), p=0.02 + 0.5 * g.random((H, dk, dv)),
                lam0=0.5 + g.random((B, H, dk, dv)), eta0=g.standard_normal((B, H, dk, dv)))


def test_channel_independent_gates_match_per_slot_form():
    x = _inputs(0)
    B, T, H, dk = x["q"].shape
    dv = x["v"].shape[-1]
    a = np.repeat(x["a"][:, :, :1], dv, 2)
    p = np.repeat(x["p"][:, :, :1], dv, 2)
    at = np.broadcast_to(a[..., 0], (B, T, H, dk)).copy()
    pt = np.broadcast_to(p[..., 0], (B, T, H, dk)).copy()
    f1 = oracle.forward_nd(x["q"], x["k"], x["v"], a, p, x["r"], x["lam0"], x["eta0"])
    f0 = oracle.forward(x["q"], x["k"], x["v"], at, pt, x["r"], x["lam0"], x["eta0"])
    for n in ("y", "yvar", "lamT", "etaT"):
        np.testing.assert_allclose(f1[n], f0[n], rtol=1e-13, atol=1e-13)
    g = np.random.default_rng(1)
    dy, dyvar = g.standard_normal((B, T, H, dv)), g.standard_normal((B, T, H, dv))
    b1 = oracle.backward_nd(x["q"], x["k"], x["v"], a, p, x["r"], x["lam0"], x["eta0"], dy, dyvar=dyvar)
    b0 = oracle.backward(x["q"], x["k"], x["v"], at, pt, x["r"], x["lam0"], x["eta0"], dy, dyvar=dyvar)
    for n in ("dq", "dk", "dv", "dr", "dlam0", "deta0"):
        np.testing.assert_allclose(b1[n], b0[n], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b1["g_abar"].sum(-1), b0["da"].sum(axis=(0, 1)), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b1["g_pbar"].sum(-1), b0["dp"].sum(axis=(0, 1)), rtol=1e-12, atol=1e-12)


def test_every_element_is_a_covariance_form_kalman_filter():
    x = _inputs(2, B=1, T=15, H=1, dk=4, dv=3)
    out = oracle.forward_nd(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], x["lam0"], x["eta0"])
    Sig = 1.0 / x["lam0"][0, 0]
    mu = x["eta0"][0, 0] * Sig
    a, p = x["a"][0], x["p"][0]
    for t in range(15):
        kt = x["k"][0, t, 0][:, None]
        rt, vt, qt = x["r"][0, t, 0][None, :], x["v"][0, t, 0][None, :], x["q"][0, t, 0][:, None]
        mp = a * mu
        Sp = a * a * Sig + p
        K = Sp * kt / (kt * kt * Sp + 1.0 / rt)
        mu = mp + K * (vt - kt * mp)
        Sig = (1.0 - K * kt) * Sp
        np.testing.assert_allclose(out["y"][0, t, 0], (qt * mu).sum(0), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(out["yvar"][0, t, 0], (qt * qt * Sig).sum(0), rtol=1e-10)
    np.testing.assert_allclose(out["lamT"][0, 0], 1.0 / Sig, rtol=1e-10)
    np.testing.assert_allclose(out["etaT"][0, 0], mu / Sig, rtol=1e-10, atol=1e-12)


def _fd(loss, x, idx, h=1e-6):
    old = x[idx]
    x[idx] = old + h
    lp = loss()
    x[idx] = old - h
    lm = loss()
    x[idx] = old
    return (lp - lm) / (2 * h)


def test_gradients_finite_differences():
    x = _inputs(3, B=1, T=6, H=1, dk=2, dv=3)
    g = np.random.default_rng(4)
    B, T, H, dk = x["q"].shape
    dv = x["v"].shape[-1]
    dy, dyvar = g.standard_normal((B, T, H, dv)), g.standard_normal((B, T, H, dv))
    dlamT, detaT = g.standard_normal((B, H, dk, dv)), g.standard_normal((B, H, dk, dv))

    def loss():
        o = oracle.forward_nd(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], x["lam0"], x["eta0"])
        return float((o["y"] * dy).sum() + (o["yvar"] * dyvar).sum() + (o["lamT"] * dlamT).sum()
                     + (o["etaT"] * detaT).sum())

    gr = oracle.backward_nd(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], x["lam0"], x["eta0"], dy, dlamT,
                            detaT, dyvar)
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("r", "dr"), ("a", "g_abar"), ("p", "g_pbar"),
                        ("lam0", "dlam0"), ("eta0", "deta0")):
        for idx in np.ndindex(x[name].shape):
            fd = _fd(loss, x[name], idx)
            assert abs(fd - gr[gname][idx]) < 2e-6 * max(1.0, abs(fd)), (name, idx, fd, gr[gname][idx])


def test_ou_parameter_gradients_finite_differences_and_masses():
    x = _inputs(5, B=2, T=5, H=1, dk=2, dv=2)
    g = np.random.default_rng(6)
    H, dk, dv = x["a"].shape
    P = {"a": 1.0 + 5.0 * g.random((H, dk, dv)), "p": 0.5 + g.random((H, dk, dv)),
         "delta": 0.01 + 0.09 * g.random((H, dk, dv))}
    dy = g.standard_normal(x["v"].shape)

    def loss():
        o = oracle.forward_ou_nd(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"])
        return float((o["y"] * dy).sum())

    gr = oracle.backward_ou_nd(x["q"], x["k"], x["v"], P["a"], P["p"], P["delta"], x["r"], None, None, dy)
    for name, gname in (("a", "da"), ("p", "dp"), ("delta", "ddelta")):
        for idx in np.ndindex(P[name].shape):
            fd = _fd(loss, P[name], idx)
            assert abs(fd - gr[gname][idx]) < 2e-6 * max(1.0, abs(fd)), (name, idx, fd, gr[gname][idx])
        assert np.all(gr["mass_" + gname] >= np.abs(gr[gname]) - 1e-12)
    one = {k: v[:1, :1] for k, v in x.items() if k in ("q", "k", "v", "r")}
    g1 = oracle.backward_ou_nd(one["q"], one["k"], one["v"], P["a"], P["p"], P["delta"], one["r"], None, None,
                               dy[:1, :1])
    for gname in ("da", "dp", "ddelta"):     # a single (b, t) term: the mass is its magnitude
        np.testing.assert_allclose(g1["mass_" + gname], np.abs(g1[gname]), rtol=1e-12, atol=1e-15)
