"""Pins of the Monte Carlo readout oracle (oracle/mc.py), CPU only.

* Philox4x64-10 written out from its definition equals numpy's Philox bit
  generator (a library routine of the same published algorithm; numpy advances
  the counter before its first block, so its block i is counter i + 1).
* The draws: Box-Muller pairs satisfy z_even^2 + z_odd^2 = -2 ln(uniform); the
  normals pass a Kolmogorov-Smirnov test against N(0, 1) with the right moments;
  sampled readouts have mean ymu and variance yvar per channel.
* The loss: S = 1 reduces to cross-entropy (-logp), and the logsumexp form
  (eq. nmll_logsumexp) equals the Monte Carlo average of the likelihoods
  (eq. nmll_integral) computed directly.
* Both backward functions against central finite differences.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import mc


@pytest.mark.parametrize("key", [(0, 0), (12345, 678), (2**64 - 1, 2**63 + 5)])
def test_philox_equals_numpy(key):
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.zeros(4, dtype=np.uint64))
    raw = bg.random_raw(4 * 64).reshape(64, 4)
    ours = mc.philox4x64(np.arange(1, 65, dtype=np.uint64), key[0], key[1])
    np.testing.assert_array_equal(ours, raw)


def test_box_muller_pairs():
    e = np.arange(4096)
    z = mc.normals(e, seed=3).reshape(-1, 8)
    words = mc.philox4x64(np.arange(512, dtype=np.uint64), 3)
    u = np.stack([words & np.uint64(0xFFFFFFFF), words >> np.uint64(32)], axis=-1).reshape(-1, 8)
    for p in range(4):
        r2 = -2.0 * np.log((np.floor(u[:, 2 * p].astype(np.float64) / 256.0) + 1.0) * 2.0 ** -24)
        np.testing.assert_allclose(z[:, 2 * p] ** 2 + z[:, 2 * p + 1] ** 2, r2, rtol=1e-12, atol=1e-14)


def test_normals_distribution():
    z = mc.normals(np.arange(1 << 18), seed=11)
    assert abs(z.mean()) < 5.0 / np.sqrt(z.size)
    assert abs(z.var() - 1.0) < 5.0 * np.sqrt(2.0 / z.size)
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # consecutive elements (one Box-Muller pair, and neighbouring blocks) are uncorrelated
    assert abs(np.corrcoef(z[0::2], z[1::2])[0, 1]) < 5.0 / np.sqrt(z.size / 2)
    assert abs(np.corrcoef(z[:-8], z[8:])[0, 1]) < 5.0 / np.sqrt(z.size)


def test_sample_moments():
    g = np.random.default_rng(0)
    ymu = g.standard_normal((1, 2, 1, 16))
    yvar = np.array([[[0.25], [4.0]]])
    S = 20000
    ys = mc.mc_sample(ymu, yvar, S, seed=5)
    np.testing.assert_allclose(ys.mean(axis=0), ymu, atol=6 * np.sqrt(4.0 / S))
    var = ys.var(axis=0)
    np.testing.assert_allclose(var[:, 0], 0.25, rtol=6 * np.sqrt(2.0 / S))
    np.testing.assert_allclose(var[:, 1], 4.0, rtol=6 * np.sqrt(2.0 / S))


def test_nll_reduces_to_cross_entropy_and_matches_average():
    g = np.random.default_rng(1)
    logp = -np.abs(g.standard_normal((1, 50))) * 3
    np.testing.assert_allclose(mc.mc_nll(logp), -logp[0], rtol=1e-14)
    logp = -np.abs(g.standard_normal((10, 50))) * 3
    direct = -np.log(np.mean(np.exp(logp), axis=0))
    np.testing.assert_allclose(mc.mc_nll(logp), direct, rtol=1e-12)
    # large magnitudes: the logsumexp form stays finite where the direct average underflows
    assert np.all(np.isfinite(mc.mc_nll(logp - 2000.0)))
    np.testing.assert_allclose(mc.mc_nll(logp - 2000.0), mc.mc_nll(logp) + 2000.0, rtol=1e-12)


def test_nll_backward_finite_differences():
    g = np.random.default_rng(2)
    logp = -np.abs(g.standard_normal((6, 7))) * 2
    dnll = g.standard_normal(7)
    grad = mc.mc_nll_backward(logp, dnll)
    h = 1e-6
    for s in range(6):
        for i in range(7):
            lp, lm = logp.copy(), logp.copy()
            lp[s, i] += h
            lm[s, i] -= h
            fd = (np.dot(dnll, mc.mc_nll(lp)) - np.dot(dnll, mc.mc_nll(lm))) / (2 * h)
            assert abs(fd - grad[s, i]) < 1e-7 * max(1.0, abs(fd))


def test_sample_backward_finite_differences():
    g = np.random.default_rng(3)
    B, T, H, dv, S = 1, 3, 2, 16, 5
    ymu = g.standard_normal((B, T, H, dv))
    yvar = 0.5 + g.random((B, T, H))
    w = g.standard_normal((S, B, T, H, dv))
    dymu, dyvar = mc.mc_sample_backward(yvar, w, seed=9)
    loss = lambda m, v: float(np.sum(w * mc.mc_sample(m, v, S, seed=9)))
    h = 1e-6
    for idx in [(0, 0, 0, 0), (0, 2, 1, 15), (0, 1, 0, 7)]:
        mp, mm = ymu.copy(), ymu.copy()
        mp[idx] += h
        mm[idx] -= h
        assert abs((loss(mp, yvar) - loss(mm, yvar)) / (2 * h) - dymu[idx]) < 1e-6
    for idx in [(0, 0, 0), (0, 2, 1), (0, 1, 0)]:
        vp, vm = yvar.copy(), yvar.copy()
        vp[idx] += h
        vm[idx] -= h
        fd = (loss(ymu, vp) - loss(ymu, vm)) / (2 * h)
        assert abs(fd - dyvar[idx]) < 1e-6 * max(1.0, abs(fd))
