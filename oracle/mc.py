"""fp64 oracle of the Monte Carlo readout of KLA+ (the log-marginal-likelihood loss).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the CPU
baseline of the benchmark, never by the product path, with which it shares no code.

The training loss (ii) of the paper's appendix (eqs. nmll_integral and
nmll_logsumexp) replaces the cross-entropy of the posterior-mean readout by the
negative log of a Monte Carlo average over S draws of the readout from the
filter's posterior:

    -log p(o_t | X)  ~  -log( (1/S) sum_s p(o_t | y_t^(s)) )
                     =  -logsumexp_s( log p(o_t | y_t^(s)) ) + log S,

with y_t^(s) = q_t z_t^(s), z_t^(s) drawn from the posterior.  Under the layer's
reading of the observation precision (one per token and head), the posterior
readout of channel d is Gaussian with mean ymu_t[d] = sum_n q_t[n] H_t[n,d] / lam_t[n]
and the variance yvar_t = sum_n q_t[n]^2 / lam_t[n] shared by the channels (the
slots being independent a posteriori), so a draw is

    y^(s)[b,t,h,d] = ymu[b,t,h,d] + sqrt(yvar[b,t,h]) eps[s,b,t,h,d],  eps ~ N(0, 1).

The decoder p(o_t | y) belongs to the model; the loss is taken here from the
decoder's log-probabilities of the target tokens, logp [S, n].

Random numbers: eps is drawn by the counter-based generator Philox4x64-10 (Salmon,
Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011),
written out below from that definition, and the Box-Muller transform.  For the flat
index e of [S, B, T, H, dv], block j = e // 8 is the Philox output for counter
(j, 0, 0, 0) and key (seed, 0); its four 64-bit words w_0..w_3 give eight 32-bit
halves u_{2m} = w_m mod 2^32, u_{2m+1} = w_m div 2^32, and each pair
(u_{2p}, u_{2p+1}) the normals
    r = sqrt(-2 ln(((u_{2p} >> 8) + 1) 2^-24)),  a = (u_{2p+1} >> 8) 2^-23,
    z_{2p} = r cos(pi a),  z_{2p+1} = r sin(pi a);
element e takes z_{e mod 8}.  (The 24-bit uniforms are exact in fp32 and fp64.)
"""
from __future__ import annotations

import numpy as np

_M0, _M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157      # Philox4x64 round multipliers
_W0, _W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B      # Weyl increments of the key
_MASK32 = np.uint64(0xFFFFFFFF)


def _mulhilo64(a: int, x: np.ndarray):
    """(high, low) 64-bit halves of the 128-bit product a * x, x a uint64 array."""
    a_lo, a_hi = np.uint64(a & 0xFFFFFFFF), np.uint64(a >> 32)
    x_lo, x_hi = x & _MASK32, x >> np.uint64(32)
    ll = a_lo * x_lo
    lh = a_lo * x_hi
    hl = a_hi * x_lo
    hh = a_hi * x_hi
    mid = (ll >> np.uint64(32)) + (lh & _MASK32) + (hl & _MASK32)
    lo = (ll & _MASK32) | ((mid & _MASK32) << np.uint64(32))
    hi = hh + (lh >> np.uint64(32)) + (hl >> np.uint64(32)) + (mid >> np.uint64(32))
    return hi, lo


def philox4x64(counter0: np.ndarray, key0: int, key1: int = 0, rounds: int = 10) -> np.ndarray:
    """Philox4x64-R of the counters (counter0, 0, 0, 0): [len, 4] uint64 words."""
    x0 = np.asarray(counter0, dtype=np.uint64).copy()
    x1 = np.zeros_like(x0)
    x2 = np.zeros_like(x0)
    x3 = np.zeros_like(x0)
    k0, k1 = int(key0) & 0xFFFFFFFFFFFFFFFF, int(key1) & 0xFFFFFFFFFFFFFFFF
    with np.errstate(over="ignore"):
        for _ in range(rounds):
            hi0, lo0 = _mulhilo64(_M0, x0)
            hi1, lo1 = _mulhilo64(_M1, x2)
            x0, x1, x2, x3 = hi1 ^ x1 ^ np.uint64(k0), lo1, hi0 ^ x3 ^ np.uint64(k1), lo0
            k0 = (k0 + _W0) & 0xFFFFFFFFFFFFFFFF
            k1 = (k1 + _W1) & 0xFFFFFFFFFFFFFFFF
    return np.stack([x0, x1, x2, x3], axis=-1)


def normals(e: np.ndarray, seed: int) -> np.ndarray:
    """eps for the flat indices e (any shape), in fp64."""
    e = np.asarray(e, dtype=np.int64)
    words = philox4x64((e // 8).astype(np.uint64).ravel(), seed)        # [n, 4]
    halves = np.stack([words & _MASK32, words >> np.uint64(32)], axis=-1).reshape(-1, 8)   # u_0..u_7
    lane = (e % 8).ravel()
    pair = lane // 2
    u_r = halves[np.arange(lane.size), 2 * pair].astype(np.float64)
    u_a = halves[np.arange(lane.size), 2 * pair + 1].astype(np.float64)
    r = np.sqrt(-2.0 * np.log((np.floor(u_r / 256.0) + 1.0) * 2.0 ** -24))
    ang = np.floor(u_a / 256.0) * 2.0 ** -23
    z = np.where(lane % 2 == 0, r * np.cos(np.pi * ang), r * np.sin(np.pi * ang))
    return z.reshape(e.shape)


def _eps(S: int, shape, seed: int) -> np.ndarray:
    n = int(np.prod(shape))
    return normals(np.arange(S * n, dtype=np.int64), seed).reshape((S,) + tuple(shape))


def mc_sample(ymu, yvar, S: int, seed: int) -> np.ndarray:
    """Draws y^(s) = ymu + sqrt(yvar) eps^(s): ymu [B, T, H, dv], yvar [B, T, H] -> [S, B, T, H, dv]."""
    ymu = np.asarray(ymu, dtype=np.float64)
    yvar = np.asarray(yvar, dtype=np.float64)
    return ymu[None] + np.sqrt(yvar)[None, ..., None] * _eps(S, ymu.shape, seed)


def mc_sample_backward(yvar, dys, seed: int):
    """Gradients of a loss with respect to ymu and yvar from its gradient dys with respect
    to the draws: dymu = sum_s dys^(s), dyvar = sum_{s, d} dys^(s) eps^(s) / (2 sqrt(yvar))."""
    yvar = np.asarray(yvar, dtype=np.float64)
    dys = np.asarray(dys, dtype=np.float64)
    S = dys.shape[0]
    eps = _eps(S, dys.shape[1:], seed)
    dymu = dys.sum(axis=0)
    dyvar = (dys * eps).sum(axis=(0, 4)) / (2.0 * np.sqrt(yvar))
    return dymu, dyvar


def mc_nll(logp) -> np.ndarray:
    """-logsumexp_s(logp[s]) + log S for logp [S, n] (eq. nmll_logsumexp): [n]."""
    logp = np.asarray(logp, dtype=np.float64)
    S = logp.shape[0]
    m = logp.max(axis=0)
    return -(m + np.log(np.exp(logp - m).sum(axis=0))) + np.log(S)


def mc_nll_backward(logp, dnll) -> np.ndarray:
    """Gradient with respect to logp [S, n]: -dnll softmax_s(logp)."""
    logp = np.asarray(logp, dtype=np.float64)
    m = logp.max(axis=0)
    w = np.exp(logp - m)
    return -np.asarray(dnll, dtype=np.float64)[None] * w / w.sum(axis=0)
