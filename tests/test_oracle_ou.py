"""Pins of the oracle's OU parameterisation (Sec. 4.1, eq. discretisation).

The decay and process-noise variance of the exactly discretised OU prior are
checked against what fixes them independently of the closed form:
  * a Monte Carlo simulation of the OU stochastic differential equation
    dz = -a z dt + p dW by Euler-Maruyama with fine sub-steps (mean and variance
    of z after one step delta);
  * the transition semigroup: one step of delta1 + delta2 equals a step of delta1
    followed by one of delta2;
  * the limits: variance p^2 delta for a small step, the stationary variance
    p^2 / (2 a) for a long one, and the exact value abar = 1/2 at a delta = ln 2;
  * central finite differences of the whole filter's loss with respect to a, p
    and delta, for the reduction over (b, t) and the chain rule.
Planted mistakes in a copy of the oracle's Python module must fail these pins.
"""
import importlib.util
import os
import shutil

import numpy as np
import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _simulate_ou(a, p, delta, z0, npath, nsub, seed):
    g = np.random.default_rng(seed)
    h = delta / nsub
    z = np.full(npath, float(z0))
    for _ in range(nsub):
        z = z - a * z * h + p * np.sqrt(h) * g.standard_normal(npath)
    return z


OU_CASES = [(2.0, 1.5, 0.5), (0.3, 0.7, 2.0), (8.0, 2.0, 0.05)]


def _sde_battery(orc) -> bool:
    """True when the closed form agrees with the simulated SDE in every case."""
    ok = True
    for i, (a, p, d) in enumerate(OU_CASES):
        abar, pbar = (float(x[0, 0]) for x in orc.ou_discretise([[a]], [[p]], [[d]]))
        mean = _simulate_ou(a, p, d, 1.0, 100_000, 200, seed=10 + i).mean()
        var = _simulate_ou(a, p, d, 0.0, 100_000, 200, seed=20 + i).var()
        ok &= abs(mean - abar) <= 0.02 * abar + 0.005
        ok &= abs(var - pbar) <= 0.03 * pbar
    return bool(ok)


def test_discretisation_matches_simulated_sde():
    assert _sde_battery(O)


def test_transition_semigroup():
    g = np.random.default_rng(3)
    a = g.uniform(0.1, 10.0, (4, 5))
    p = g.uniform(0.1, 3.0, (4, 5))
    d1 = g.uniform(1e-3, 1.0, (4, 5))
    d2 = g.uniform(1e-3, 1.0, (4, 5))
    a1, p1 = O.ou_discretise(a, p, d1)
    a2, p2 = O.ou_discretise(a, p, d2)
    a12, p12 = O.ou_discretise(a, p, d1 + d2)
    np.testing.assert_allclose(a12, a1 * a2, rtol=1e-13)
    np.testing.assert_allclose(p12, a2 * a2 * p1 + p2, rtol=1e-12)


def test_limits_and_exact_value():
    a = np.array([[0.5, 3.0]])
    p = np.array([[1.2, 0.4]])
    _, small = O.ou_discretise(a, p, np.full_like(a, 1e-9))
    np.testing.assert_allclose(small / 1e-9, p * p, rtol=1e-8)
    abar_long, big = O.ou_discretise(a, p, np.full_like(a, 200.0))
    np.testing.assert_allclose(big, p * p / (2 * a), rtol=1e-12)
    assert np.all(abar_long < 1e-40)
    half, pb = O.ou_discretise([[np.log(2.0)]], [[2.0]], [[1.0]])
    assert half[0, 0] == pytest.approx(0.5, rel=1e-15)
    # 1 - abar^2 = 3/4 of the stationary variance p^2 / (2 a)
    assert pb[0, 0] == pytest.approx(0.75 * 4.0 / (2 * np.log(2.0)), rel=1e-14)


def _ou_case(seed=5):
    g = np.random.default_rng(seed)
    B, T, H, dk, dv = 2, 9, 2, 3, 2
    q, k = g.standard_normal((2, B, T, H, dk))
    v = g.standard_normal((B, T, H, dv))
    r = 0.3 + g.random((B, T, H))
    a = g.uniform(0.5, 4.0, (H, dk))
    p = g.uniform(0.3, 2.0, (H, dk))
    d = g.uniform(0.02, 0.5, (H, dk))
    lam0 = 0.5 + g.random((B, H, dk))
    eta0 = g.standard_normal((B, H, dk, dv))
    dy = g.standard_normal((B, T, H, dv))
    dlamT = g.standard_normal((B, H, dk))
    detaT = g.standard_normal((B, H, dk, dv))
    return q, k, v, a, p, d, r, lam0, eta0, dy, dlamT, detaT


def _fd_battery(orc) -> bool:
    """True when the oracle's (da, dp, ddelta) match central differences of the loss."""
    q, k, v, a, p, d, r, lam0, eta0, dy, dlamT, detaT = _ou_case()

    def loss(a_, p_, d_):
        o = orc.forward_ou(q, k, v, a_, p_, d_, r, lam0, eta0, nthreads=1)
        return float((o["y"] * dy).sum() + (o["lamT"] * dlamT).sum() + (o["etaT"] * detaT).sum())

    g = orc.backward_ou(q, k, v, a, p, d, r, lam0, eta0, dy, dlamT, detaT, nthreads=1)
    ok = True
    for name, idx in (("da", 0), ("dp", 1), ("ddelta", 2)):
        base = [a, p, d]
        fd = np.zeros_like(base[idx])
        for i in np.ndindex(fd.shape):
            h = 1e-6 * max(1.0, abs(base[idx][i]))
            plus = [x.copy() for x in base]
            minus = [x.copy() for x in base]
            plus[idx][i] += h
            minus[idx][i] -= h
            fd[i] = (loss(*plus) - loss(*minus)) / (2 * h)
        err = np.max(np.abs(g[name] - fd)) / max(np.max(np.abs(fd)), 1e-12)
        ok &= err < 1e-6
    return bool(ok)


def test_ou_gradients_match_central_differences():
    assert _fd_battery(O)


def test_ou_decode_step_equals_forward_token():
    q, k, v, a, p, d, r, lam0, eta0, *_ = _ou_case(seed=8)
    one = O.forward_ou(q[:, :1], k[:, :1], v[:, :1], a, p, d, r[:, :1], lam0, eta0, nthreads=1)
    dec = O.decode_step_ou(q[:, 0], k[:, 0], v[:, 0], a, p, d, r[:, 0], lam0, eta0)
    np.testing.assert_allclose(dec["y"], one["y"][:, 0], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(dec["lam"], one["lamT"], rtol=1e-14)


# ---- planted mistakes, each in a copy of the oracle's Python module
OU_MUTATIONS = {
    "variance_rate_not_doubled": ("pbar = p * p * (-np.expm1(-2.0 * a * delta)) / (2.0 * a)",
                                  "pbar = p * p * (-np.expm1(-1.0 * a * delta)) / (2.0 * a)"),
    "variance_scale_missing_half": ("pbar = p * p * (-np.expm1(-2.0 * a * delta)) / (2.0 * a)",
                                    "pbar = p * p * (-np.expm1(-2.0 * a * delta)) / a"),
    "decay_half_rate": ("abar = np.exp(-a * delta)\n    pbar", "abar = np.exp(-a * delta * 0.5)\n    pbar"),
    "vjp_step_term_dropped": ("ddelta = g_abar * (-a * abar) + g_pbar * p * p * E",
                              "ddelta = g_abar * (-a * abar)"),
    "vjp_rate_sign": ("(delta * E - s) / a", "(delta * E + s) / a"),
    "vjp_scale_factor": ("dp = g_pbar * 2.0 * p * s", "dp = g_pbar * p * s"),
}


def _load_mutant(tmp_path, name):
    old, new = OU_MUTATIONS[name]
    src = open(os.path.join(ROOT, "oracle", "__init__.py")).read()
    assert src.count(old) == 1, f"mutation anchor not unique/present: {old}"
    mut_dir = tmp_path / name
    mut_dir.mkdir()
    (mut_dir / "__init__.py").write_text(src.replace(old, new))
    # the C part is unchanged: reuse the built library
    shutil.copy(O._LIB_PATH, mut_dir / "_kla_oracle.so")
    spec = importlib.util.spec_from_file_location(f"oracle_ou_{name}", mut_dir / "__init__.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", sorted(OU_MUTATIONS))
def test_planted_ou_mistake_is_caught(tmp_path, name):
    O._load()   # the library the copies reuse exists
    mod = _load_mutant(tmp_path, name)
    assert not (_sde_battery(mod) and _fd_battery(mod)), f"mutation {name} passed the pins"
