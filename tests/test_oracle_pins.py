"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's recursion: each reaches the same
quantity by another route (the textbook covariance-form Kalman filter, the
Moebius / affine composition of Corollaries 1-2 evaluated in a tree order, the
Riccati fixed point, the closed form at zero process noise, the moment-form
recursion, the ridge objective minimised numerically, the unrolled attention
matrix, a hand-derived fixture, and central finite differences).
"""
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy.optimize import minimize_scalar

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _case(T, dk, dv, seed, per_channel=True, p_scale=1.0):
    g = np.random.default_rng(seed)
    k = g.standard_normal((T, dk)) * 0.7
    q = g.standard_normal((T, dk))
    v = g.standard_normal((T, dv))
    a = 1.0 / (1.0 + np.exp(-(g.standard_normal((T, dk)) + 1.5)))
    p = np.log1p(np.exp(g.standard_normal((T, dk)) - 1.0)) * p_scale
    r = np.log1p(np.exp(g.standard_normal((T, dv) if per_channel else (T, 1))))
    r = np.broadcast_to(r, (T, dv)).copy()
    lam0 = 0.5 + g.random((dk, dv))
    eta0 = g.standard_normal((dk, dv))
    return dict(q=q, k=k, v=v, a=a, p=p, r=r, lam0=lam0, eta0=eta0)


def _fwd(c):
    """Oracle forward on a single sequence given as [T, *] arrays."""
    out = oracle.forward(c["q"][None, :, None], c["k"][None, :, None], c["v"][None, :, None],
                         c["a"][None, :, None], c["p"][None, :, None], c["r"][None, :, None],
                         c["lam0"][None, None], c["eta0"][None, None])
    return out["y"][0, :, 0], out["yvar"][0, :, 0], out["lamT"][0, 0], out["etaT"][0, 0]


# ---------------------------------------------------------------- golden
def test_hand_derived_three_steps():
    rows = {}
    table = []
    for line in open(os.path.join(GOLDEN, "scalar_three_steps.txt")):
        line = line.split("#")[0].split()
        if not line:
            continue
        if line[0].isalpha():
            rows[line[0]] = [int(x) for x in line[1:]]
        else:
            table.append([int(x) for x in line])
    fr = lambda xs: float(Fraction(xs[0], xs[1]))
    a, p, k, Lv, qv = (fr(rows[n]) for n in ("abar", "pbar", "k", "Lv", "q"))
    v = np.array(rows["v"], dtype=float)
    T = len(v)
    one = lambda x: np.full((T, 1), x)
    lt, et = oracle.trace(one(k), v[:, None], one(a), one(p), one(Lv), 1.0, 0.0)
    c = dict(q=one(qv), k=one(k), v=v[:, None], a=one(a), p=one(p), r=one(Lv),
             lam0=np.ones((1, 1)), eta0=np.zeros((1, 1)))
    y, yvar, _, _ = _fwd(c)
    for t, ln, ld, en, ed, yn, yd, wn, wd in table:
        assert lt[t, 0, 0] == pytest.approx(ln / ld, rel=1e-15)
        assert et[t, 0, 0] == pytest.approx(en / ed, rel=1e-15)
        assert y[t - 1, 0] == pytest.approx(yn / yd, rel=1e-15)
        assert yvar[t - 1, 0] == pytest.approx(wn / wd, rel=1e-15)


# ------------------------------------------- covariance-form Kalman filter
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_matches_covariance_form_kalman_filter(seed):
    T, dk, dv = 40, 3, 2
    c = _case(T, dk, dv, seed)
    lt, et = oracle.trace(c["k"], c["v"], c["a"], c["p"], c["r"], c["lam0"], c["eta0"])
    y, yvar, _, _ = _fwd(c)
    # textbook moment-form filter, one scalar per (n, d) (Kalman filter column of
    # the KF/IF comparison table, diagonal case)
    Sig = 1.0 / c["lam0"]
    mu = c["eta0"] / c["lam0"]
    for t in range(T):
        a, p, k = c["a"][t][:, None], c["p"][t][:, None], c["k"][t][:, None]
        r, v = c["r"][t][None, :], c["v"][t][None, :]
        mu_pred = a * mu
        S_pred = a * a * Sig + p
        K = S_pred * k / (k * k * S_pred + 1.0 / r)
        mu = mu_pred + K * (v - k * mu_pred)
        Sig = (1.0 - K * k) * S_pred
        np.testing.assert_allclose(lt[t + 1], 1.0 / Sig, rtol=1e-12)
        np.testing.assert_allclose(et[t + 1] / lt[t + 1], mu, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(y[t], (c["q"][t][:, None] * mu).sum(0), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(yvar[t], (c["q"][t][:, None] ** 2 * Sig).sum(0), rtol=1e-12)


# --------------------------------------- Moebius composition (Thm 1, Cor 1)
def test_mobius_matrix_entries_and_invariants():
    g = np.random.default_rng(5)
    for _ in range(50):
        k, q_, p, r = g.standard_normal(), g.random(), g.random(), g.random() + 0.1
        a = g.random() * 0.99 + 0.01
        M = oracle.mobius_matrix(k, a, p, r)
        assert np.all(M >= 0)
        assert np.linalg.det(M) == pytest.approx(a * a, rel=1e-12)
        lam = g.random() * 5 + 0.01
        # the Moebius action equals one predict/update of the covariance form
        S_pred = a * a / lam + p
        assert oracle.mobius_apply(M, lam) == pytest.approx(1.0 / S_pred + k * k * r, rel=1e-13)


def test_mobius_prefix_reproduces_recursion():
    T, dk, dv = 48, 2, 3
    c = _case(T, dk, dv, 7)
    lt, _ = oracle.trace(c["k"], c["v"], c["a"], c["p"], c["r"], c["lam0"], c["eta0"])
    for n in range(dk):
        for d in range(dv):
            P = np.eye(2)
            for t in range(T):
                M = oracle.mobius_matrix(c["k"][t, n], c["a"][t, n], c["p"][t, n], c["r"][t, d])
                P = oracle.mobius_compose(M, P)
                assert oracle.mobius_apply(P, c["lam0"][n, d]) == pytest.approx(lt[t + 1, n, d], rel=1e-12)


def test_compose_is_matrix_product():
    g = np.random.default_rng(11)
    for _ in range(20):
        A, B = g.random((2, 2)), g.random((2, 2))
        np.testing.assert_allclose(oracle.mobius_compose(A, B), A @ B, rtol=1e-15)


def _proj(M):
    return M / np.abs(M).max()


def test_mobius_compose_associative_random_triples():
    g = np.random.default_rng(3)
    for _ in range(200):
        Ms = [oracle.mobius_matrix(g.standard_normal(), g.random() * 0.98 + 0.02,
                                   g.random() * 2, g.random() * 3 + 0.05) for _ in range(3)]
        L = oracle.mobius_compose(oracle.mobius_compose(Ms[2], Ms[1]), Ms[0])
        R = oracle.mobius_compose(Ms[2], oracle.mobius_compose(Ms[1], Ms[0]))
        np.testing.assert_allclose(_proj(L), _proj(R), rtol=1e-13, atol=1e-15)
        lam = g.random() * 4 + 0.01
        seq = oracle.mobius_apply(Ms[2], oracle.mobius_apply(Ms[1], oracle.mobius_apply(Ms[0], lam)))
        assert oracle.mobius_apply(L, lam) == pytest.approx(seq, rel=1e-13)


def test_affine_compose_associative_random_triples():
    g = np.random.default_rng(4)
    for _ in range(100):
        dk, dv = 4, 3
        fs = [g.random(dk) * 1.5 for _ in range(3)]
        bs = [g.standard_normal((dk, dv)) for _ in range(3)]
        f21, b21 = oracle.affine_compose(fs[2], bs[2], fs[1], bs[1])
        fL, bL = oracle.affine_compose(f21, b21, fs[0][:, None], bs[0])
        f10, b10 = oracle.affine_compose(fs[1], bs[1], fs[0], bs[0])
        fR, bR = oracle.affine_compose(fs[2][:, None], bs[2], f10, b10)
        np.testing.assert_allclose(fL, fR, rtol=1e-14)
        np.testing.assert_allclose(bL, bR, rtol=1e-13, atol=1e-14)
        # applying the composed map equals applying the three maps in turn
        x = g.standard_normal((dk, dv))
        y = x
        for f, b in zip(fs, bs):
            y = f[:, None] * y + b
        np.testing.assert_allclose(fL * x + bL, y, rtol=1e-12, atol=1e-13)


# ------------------------------------------------ tree-ordered scans (T<=64)
def _blelloch_exclusive(items, combine, identity):
    """Work-efficient up-sweep / down-sweep exclusive scan; n a power of two."""
    n = len(items)
    x = list(items)
    step = 1
    while step < n:
        for i in range(2 * step - 1, n, 2 * step):
            x[i] = combine(x[i], x[i - step])          # later element on the left
        step *= 2
    x[n - 1] = identity
    step = n // 2
    while step >= 1:
        for i in range(2 * step - 1, n, 2 * step):
            left = x[i - step]
            x[i - step] = x[i]
            x[i] = combine(left, x[i])
        step //= 2
    return x


def _random_tree_product(items, combine, g):
    """Combine a list in a random bracketing (order of the list is kept)."""
    xs = list(items)
    while len(xs) > 1:
        i = int(g.integers(0, len(xs) - 1))
        xs[i:i + 2] = [combine(xs[i + 1], xs[i])]
    return xs[0]


@pytest.mark.parametrize("T", [1, 7, 32, 64])
def test_sequential_equals_tree_ordered_scan(T):
    dk, dv = 2, 2
    c = _case(T, dk, dv, 100 + T)
    lt, et = oracle.trace(c["k"], c["v"], c["a"], c["p"], c["r"], c["lam0"], c["eta0"])
    npow = 1 << max(0, (T - 1).bit_length())
    g = np.random.default_rng(T)
    for n in range(dk):
        for d in range(dv):
            Ms = [oracle.mobius_matrix(c["k"][t, n], c["a"][t, n], c["p"][t, n], c["r"][t, d])
                  for t in range(T)] + [np.eye(2)] * (npow - T)
            excl = _blelloch_exclusive(Ms, oracle.mobius_compose, np.eye(2))
            incl = [oracle.mobius_compose(Ms[t], excl[t]) for t in range(T)]
            lam = np.array([oracle.mobius_apply(P, c["lam0"][n, d]) for P in incl])
            np.testing.assert_allclose(lam, lt[1:, n, d], rtol=1e-12)
            # random bracketing of the whole product
            P = _random_tree_product(Ms[:T], oracle.mobius_compose, g)
            assert oracle.mobius_apply(P, c["lam0"][n, d]) == pytest.approx(lt[T, n, d], rel=1e-12)
            # affine scan of the information mean, gates from the scanned precisions
            lam_prev = np.concatenate([[c["lam0"][n, d]], lam[:-1]])
            f = c["a"][:, n] / (c["a"][:, n] ** 2 + c["p"][:, n] * lam_prev)
            b = c["k"][:, n] * c["r"][:, d] * c["v"][:, d]
            pairs = [(np.array([f[t]]), np.array([b[t]])) for t in range(T)] + \
                    [(np.ones(1), np.zeros(1))] * (npow - T)
            comb = lambda x2, x1: oracle.affine_compose(x2[0], x2[1], x1[0], x1[1])
            excl = _blelloch_exclusive(pairs, comb, (np.ones(1), np.zeros(1)))
            for t in range(T):
                F, Bv = comb(pairs[t], excl[t])
                assert F[0] * c["eta0"][n, d] + Bv[0] == pytest.approx(et[t + 1, n, d], rel=1e-11, abs=1e-13)
            F, Bv = _random_tree_product(pairs[:T], comb, g)
            assert F[0] * c["eta0"][n, d] + Bv[0] == pytest.approx(et[T, n, d], rel=1e-11, abs=1e-13)


# ------------------------------------------------------ steady state
@pytest.mark.parametrize("a,p,k,r,v", [(0.9, 0.05, 0.3, 0.8, 1.3), (0.5, 1.0, 1.0, 1.0, -0.7),
                                       (0.99, 0.001, 0.1, 2.0, 0.4)])
def test_riccati_fixed_point(a, p, k, r, v):
    T = 6000
    one = lambda x: np.full((T, 1), x)
    lt, et = oracle.trace(one(k), one(v), one(a), one(p), one(r), 1.0, 0.0)
    phi = k * k * r
    # lam = lam/(a^2 + p lam) + phi  <=>  p lam^2 + (a^2 - 1 - p phi) lam - a^2 phi = 0
    B = a * a - 1 - p * phi
    lam_star = (-B + np.sqrt(B * B + 4 * p * a * a * phi)) / (2 * p)
    f_star = a / (a * a + p * lam_star)
    eta_star = k * r * v / (1 - f_star)
    assert lt[-1, 0, 0] == pytest.approx(lam_star, rel=1e-12)
    assert et[-1, 0, 0] / lt[-1, 0, 0] == pytest.approx(eta_star / lam_star, rel=1e-10)


# ------------------------------------- zero process noise: closed form
def test_zero_process_noise_closed_form():
    T, dk, dv = 50, 3, 2
    g = np.random.default_rng(9)
    a_n = 0.9 + 0.09 * g.random(dk)            # constant per slot
    k_n = g.standard_normal(dk)
    r = np.log1p(np.exp(g.standard_normal((T, dv))))
    v = g.standard_normal((T, dv))
    lam0 = 0.5 + g.random((dk, dv))
    eta0 = g.standard_normal((dk, dv))
    A = np.tile(a_n, (T, 1))
    K = np.tile(k_n, (T, 1))
    lt, et = oracle.trace(K, v, A, np.zeros((T, dk)), r, lam0, eta0)
    for t in range(1, T + 1):
        s = np.arange(1, t + 1)
        w2 = a_n[:, None] ** (-2.0 * (t - s))[None, :]          # [dk, t]
        w1 = a_n[:, None] ** (-1.0 * (t - s))[None, :]
        lam = a_n[:, None] ** (-2.0 * t) * lam0 + k_n[:, None] ** 2 * (w2 @ r[:t])
        eta = a_n[:, None] ** (-1.0 * t) * eta0 + k_n[:, None] * (w1 @ (r[:t] * v[:t]))
        np.testing.assert_allclose(lt[t], lam, rtol=1e-11)
        np.testing.assert_allclose(et[t], eta, rtol=1e-10, atol=1e-12)


# ------------------------------------ moment form and ridge objective
def test_moment_form_and_ridge_argmin():
    T, dk, dv = 30, 2, 2
    c = _case(T, dk, dv, 21)
    lt, et = oracle.trace(c["k"], c["v"], c["a"], c["p"], c["r"], c["lam0"], c["eta0"])
    mu_or = et / lt
    # precisions from the Moebius product (independent of the oracle's recursion)
    mu = c["eta0"] / c["lam0"]
    lam = c["lam0"].copy()
    for t in range(T):
        a, p, k = c["a"][t][:, None], c["p"][t][:, None], c["k"][t][:, None]
        r, v = c["r"][t][None, :], c["v"][t][None, :]
        lam_new = np.empty_like(lam)
        for n in range(dk):
            for d in range(dv):
                M = np.array([[1 + p[n, 0] * k[n, 0] ** 2 * r[0, d], a[n, 0] ** 2 * k[n, 0] ** 2 * r[0, d]],
                              [p[n, 0], a[n, 0] ** 2]])
                lam_new[n, d] = (M[0, 0] * lam[n, d] + M[0, 1]) / (M[1, 0] * lam[n, d] + M[1, 1])
        # Corollary (moment form): gated recurrence of the posterior mean
        phi = k * k * r
        mu_mf = a * (1 - phi / lam_new) * mu + k * r * v / lam_new
        np.testing.assert_allclose(mu_or[t + 1], mu_mf, rtol=1e-10, atol=1e-12)
        # eq. kla-ridge: the same mean minimises the precision-weighted objective
        prior_prec = lam / (a * a + p * lam)
        for n in range(dk):
            for d in range(dv):
                L = lambda m: r[0, d] * (v[0, d] - k[n, 0] * m) ** 2 + \
                    prior_prec[n, d] * (m - a[n, 0] * mu[n, d]) ** 2
                res = minimize_scalar(L, bracket=(-10, 10), tol=1e-14)
                assert res.x == pytest.approx(mu_or[t + 1, n, d], rel=1e-6, abs=1e-7)
        mu, lam = mu_mf, lam_new


# ------------------------------------------- unrolled attention matrix
def test_unrolled_attention_matrix():
    T, dk, dv = 24, 3, 2
    c = _case(T, dk, dv, 33)
    lt, _ = oracle.trace(c["k"], c["v"], c["a"], c["p"], c["r"], c["lam0"], c["eta0"])
    y, _, _, _ = _fwd(c)
    lam = lt[1:]
    lam_prev = lt[:-1]
    f = c["a"][:, :, None] / (c["a"][:, :, None] ** 2 + c["p"][:, :, None] * lam_prev)   # [T, dk, dv]
    y_bf = np.zeros((T, dv))
    for i in range(T):
        for j in range(i + 1):
            W = np.prod(f[j + 1:i + 1], axis=0) * c["k"][j][:, None] * c["r"][j][None, :]   # [dk, dv]
            y_bf[i] += (c["q"][i][:, None] / lam[i] * W * c["v"][j][None, :]).sum(0)
        init = np.prod(f[:i + 1], axis=0) * c["eta0"]
        y_bf[i] += (c["q"][i][:, None] / lam[i] * init).sum(0)
    np.testing.assert_allclose(y, y_bf, rtol=1e-10, atol=1e-12)


# --------------------------------------------------- consistency checks
def test_decode_steps_equal_forward():
    B, T, H, dk, dv = 2, 9, 2, 3, 4
    g = np.random.default_rng(42)
    q, k = g.standard_normal((2, B, T, H, dk))
    v = g.standard_normal((B, T, H, dv))
    a = 0.6 + 0.4 * g.random((B, T, H, dk))
    p = g.random((B, T, H, dk))
    r = 0.1 + g.random((B, T, H))
    lam0 = 0.5 + g.random((B, H, dk))
    eta0 = g.standard_normal((B, H, dk, dv))
    ref = oracle.forward(q, k, v, a, p, r, lam0, eta0)
    lam, eta = lam0, eta0
    for t in range(T):
        st = oracle.decode_step(q[:, t], k[:, t], v[:, t], a[:, t], p[:, t], r[:, t], lam, eta)
        np.testing.assert_allclose(st["y"], ref["y"][:, t], rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(st["yvar"], ref["yvar"][:, t], rtol=1e-13)
        lam, eta = st["lam"], st["eta"]
    np.testing.assert_allclose(lam, ref["lamT"], rtol=1e-13)
    np.testing.assert_allclose(eta, ref["etaT"], rtol=1e-13, atol=1e-14)


def test_split_sequence_resume():
    B, T, H, dk, dv = 1, 20, 3, 4, 2
    g = np.random.default_rng(8)
    q, k = g.standard_normal((2, B, T, H, dk))
    v = g.standard_normal((B, T, H, dv))
    a = 0.6 + 0.4 * g.random((B, T, H, dk))
    p = g.random((B, T, H, dk))
    r = 0.1 + g.random((B, T, H))
    ref = oracle.forward(q, k, v, a, p, r)
    s = 7
    first = oracle.forward(q[:, :s], k[:, :s], v[:, :s], a[:, :s], p[:, :s], r[:, :s])
    second = oracle.forward(q[:, s:], k[:, s:], v[:, s:], a[:, s:], p[:, s:], r[:, s:],
                            first["lamT"], first["etaT"])
    np.testing.assert_allclose(np.concatenate([first["y"], second["y"]], 1), ref["y"], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(second["lamT"], ref["lamT"], rtol=1e-13)
    np.testing.assert_allclose(second["etaT"], ref["etaT"], rtol=1e-13, atol=1e-14)


def test_per_head_precision_keeps_channels_identical():
    B, T, H, dk, dv = 1, 15, 1, 3, 5
    g = np.random.default_rng(1)
    q, k = g.standard_normal((2, B, T, H, dk))
    v = g.standard_normal((B, T, H, dv))
    a = 0.6 + 0.4 * g.random((B, T, H, dk))
    p = g.random((B, T, H, dk))
    r = 0.1 + g.random((B, T, H))
    out = oracle.forward(q, k, v, a, p, np.broadcast_to(r[..., None], (B, T, H, dv)))
    assert np.all(out["lamT"] == out["lamT"][..., :1])
    assert np.all(out["yvar"] == out["yvar"][..., :1])


# --------------------------------------------- backward: finite differences
def _loss(inp, dy, dlamT, detaT, dyvar):
    out = oracle.forward(inp["q"], inp["k"], inp["v"], inp["a"], inp["p"], inp["r"],
                         inp["lam0"], inp["eta0"])
    return ((out["y"] * dy).sum() + (out["lamT"] * dlamT).sum() + (out["etaT"] * detaT).sum()
            + (out["yvar"] * dyvar).sum())


@pytest.mark.parametrize("per_head", [False, True])
def test_backward_matches_central_differences(per_head):
    B, T, H, dk, dv = 1, 7, 2, 3, 2
    g = np.random.default_rng(17 + per_head)
    inp = dict(q=g.standard_normal((B, T, H, dk)), k=g.standard_normal((B, T, H, dk)),
               v=g.standard_normal((B, T, H, dv)), a=0.5 + 0.5 * g.random((B, T, H, dk)),
               p=0.1 + g.random((B, T, H, dk)))
    if per_head:
        inp["r"] = 0.2 + g.random((B, T, H))
        inp["lam0"] = 0.5 + g.random((B, H, dk))
        dlamT = g.standard_normal((B, H, dk))
        dyvar = g.standard_normal((B, T, H))
    else:
        inp["r"] = 0.2 + g.random((B, T, H, dv))
        inp["lam0"] = 0.5 + g.random((B, H, dk, dv))
        dlamT = g.standard_normal((B, H, dk, dv))
        dyvar = g.standard_normal((B, T, H, dv))
    inp["eta0"] = g.standard_normal((B, H, dk, dv))
    dy = g.standard_normal((B, T, H, dv))
    detaT = g.standard_normal((B, H, dk, dv))
    gr = oracle.backward(inp["q"], inp["k"], inp["v"], inp["a"], inp["p"], inp["r"],
                         inp["lam0"], inp["eta0"], dy, dlamT, detaT, dyvar=dyvar)
    names = {"q": "dq", "k": "dk", "v": "dv", "a": "da", "p": "dp", "r": "dr",
             "lam0": "dlam0", "eta0": "deta0"}
    h = 1e-6
    for name, gname in names.items():
        x = inp[name]
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            old = x[idx]
            x[idx] = old + h
            lp = _loss(inp, dy, dlamT, detaT, dyvar)
            x[idx] = old - h
            lm = _loss(inp, dy, dlamT, detaT, dyvar)
            x[idx] = old
            fd[idx] = (lp - lm) / (2 * h)
        assert gr[gname].shape == x.shape, gname
        np.testing.assert_allclose(gr[gname], fd, rtol=2e-6, atol=2e-7, err_msg=gname)
