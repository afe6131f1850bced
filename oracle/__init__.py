"""fp64 CPU oracle of the Kalman Linear Attention filter.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark may import this package; the product path never does, and
it shares no code with the GPU kernels.

The arithmetic lives in ``kla_oracle.c`` (plain sequential C, double precision):
each (batch, head, key slot, value channel) runs the scalar information filter
of Theorems 1 and 2 token after token, and the readout contracts over the key
slot as in Algorithm 1.  This module only marshals numpy arrays.

Shapes follow the row-major ``[B, T, H, *]`` layout of the product:
``q, k, a, p`` are ``[B, T, H, dk]``, ``v`` is ``[B, T, H, dv]``.  The value
precision ``r`` may be ``[B, T, H]`` (one precision per token and head, the
product's layout) or ``[B, T, H, dv]`` (one per value channel, the literal
shape in Algorithm 1).  In the first case results come back in the product's
shapes: ``yvar [B, T, H]``, ``lamT [B, H, dk]``, ``dr [B, T, H]`` and
``dlam0 [B, H, dk]``; the per-channel copies of the precision, which then all
coincide, are reduced (the final precision reads channel 0; the gradient of an
initial precision shared by all channels is the sum over channels).

The ``*_ou`` functions take the gates from time-invariant OU parameters
``a, p, delta [H, dk]`` instead (Sec. 4.1, eq. discretisation): the exact
discretisation is written out in numpy (fp64), broadcast over (b, t) and fed to
the same filter; the parameter gradients are the per-token gate gradients summed
over (b, t) and taken through the discretisation by the chain rule.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_kla_oracle.so")
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I = ctypes.c_int


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.kla_oracle_forward.argtypes = [_I] * 5 + [_D] * 12 + [_I]
    lib.kla_oracle_backward.argtypes = [_I] * 5 + [_D] * 20 + [_I]
    lib.kla_oracle_decode_step.argtypes = [_I] * 4 + [_D] * 10
    lib.kla_oracle_forward_nd.argtypes = [_I] * 5 + [_D] * 12 + [_I]
    lib.kla_oracle_backward_nd.argtypes = [_I] * 5 + [_D] * 23 + [_I]
    lib.kla_oracle_trace.argtypes = [_I] * 3 + [_D] * 9
    lib.kla_oracle_mobius_matrix.argtypes = [ctypes.c_double] * 4 + [_D]
    lib.kla_oracle_mobius_compose.argtypes = [_D] * 3
    lib.kla_oracle_mobius_apply.argtypes = [_D, ctypes.c_double]
    lib.kla_oracle_mobius_apply.restype = ctypes.c_double
    lib.kla_oracle_affine_compose.argtypes = [_I] + [_D] * 6
    for fn in ("kla_oracle_forward", "kla_oracle_backward", "kla_oracle_decode_step", "kla_oracle_forward_nd",
               "kla_oracle_backward_nd",
               "kla_oracle_trace", "kla_oracle_mobius_matrix", "kla_oracle_mobius_compose",
               "kla_oracle_affine_compose"):
        getattr(lib, fn).restype = None
    _lib = lib
    return lib


def _c(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(x: Optional[np.ndarray]):
    if x is None:
        return ctypes.cast(None, _D)
    return x.ctypes.data_as(_D)


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def _prep(q, k, v, a, p, r, lam0, eta0):
    q, k, v, a, p, r = (_c(x) for x in (q, k, v, a, p, r))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    per_head = r.ndim == 3
    if per_head:
        r = _c(np.broadcast_to(r[..., None], (B, T, H, dv)))
    if lam0 is not None:
        lam0 = _c(lam0)
        if lam0.ndim == 3:
            lam0 = _c(np.broadcast_to(lam0[..., None], (B, H, dk, dv)))
    if eta0 is not None:
        eta0 = _c(eta0)
    return q, k, v, a, p, r, lam0, eta0, (B, T, H, dk, dv), per_head


def forward(q, k, v, a, p, r, lam0=None, eta0=None, nthreads: Optional[int] = None) -> dict:
    """Sequential filter over the whole sequence; returns y, yvar, lamT, etaT."""
    lib = _load()
    q, k, v, a, p, r, lam0, eta0, (B, T, H, dk, dv), per_head = _prep(q, k, v, a, p, r, lam0, eta0)
    y = np.empty((B, T, H, dv))
    yvar = np.empty((B, T, H, dv))
    lamT = np.empty((B, H, dk, dv))
    etaT = np.empty((B, H, dk, dv))
    lib.kla_oracle_forward(B, T, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(a), _ptr(p), _ptr(r),
                           _ptr(lam0), _ptr(eta0), _ptr(y), _ptr(yvar), _ptr(lamT), _ptr(etaT),
                           nthreads or default_threads())
    if per_head:
        yvar = yvar[..., 0].copy()
        lamT = lamT[..., 0].copy()
    return {"y": y, "yvar": yvar, "lamT": lamT, "etaT": etaT}


def backward(q, k, v, a, p, r, lam0, eta0, dy, dlamT=None, detaT=None,
             nthreads: Optional[int] = None, dyvar=None) -> dict:
    """Exact reverse-mode gradient of ``forward``'s y, lamT, etaT and (with
    ``dyvar``, shaped like ``forward``'s yvar) yvar."""
    lib = _load()
    lam0_in_shape = None if lam0 is None else np.asarray(lam0).shape
    q, k, v, a, p, r, lam0, eta0, (B, T, H, dk, dv), per_head = _prep(q, k, v, a, p, r, lam0, eta0)
    dy = _c(dy)
    if dyvar is not None:
        dyvar = _c(dyvar)
        if per_head:
            # the per-head variance is channel 0 of the per-channel one: seed channel 0 only
            full = np.zeros((B, T, H, dv))
            full[..., 0] = dyvar
            dyvar = full
    if dlamT is not None:
        dlamT = _c(dlamT)
        if dlamT.ndim == 3:
            # the final precision is shared by all channels: seed channel 0 only
            full = np.zeros((B, H, dk, dv))
            full[..., 0] = dlamT
            dlamT = full
    if detaT is not None:
        detaT = _c(detaT)
    out = {n: np.empty((B, T, H, dk)) for n in ("dq", "dk", "da", "dp")}
    out["dv"] = np.empty((B, T, H, dv))
    out["dr"] = np.empty((B, T, H, dv))
    dlam0 = np.empty((B, H, dk, dv))
    deta0 = np.empty((B, H, dk, dv))
    lib.kla_oracle_backward(B, T, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(a), _ptr(p), _ptr(r),
                            _ptr(lam0), _ptr(eta0), _ptr(dy), _ptr(dyvar), _ptr(dlamT), _ptr(detaT),
                            _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["da"]),
                            _ptr(out["dp"]), _ptr(out["dr"]), _ptr(dlam0), _ptr(deta0),
                            nthreads or default_threads())
    if per_head:
        out["dr"] = out["dr"].sum(-1)
    if lam0_in_shape is not None and len(lam0_in_shape) == 3:
        dlam0 = dlam0.sum(-1)
    out["dlam0"] = dlam0
    out["deta0"] = deta0
    return out


def decode_step(q, k, v, a, p, r, lam, eta) -> dict:
    """One recurrent step on a carried belief; inputs ``[S, H, *]``.

    ``lam`` may be ``[S, H, dk]`` (shared over channels) or ``[S, H, dk, dv]``.
    Returns new copies: y, yvar, lam, eta (input arrays are not modified)."""
    lib = _load()
    q, k, v, a, p, r = (_c(x) for x in (q, k, v, a, p, r))
    S, H, dk = k.shape
    dv = v.shape[-1]
    per_head = r.ndim == 2
    if per_head:
        r = _c(np.broadcast_to(r[..., None], (S, H, dv)))
    lam = _c(lam).copy()
    lam_per_slot = lam.ndim == 3
    if lam_per_slot:
        lam = _c(np.broadcast_to(lam[..., None], (S, H, dk, dv)))
    eta = _c(eta).copy()
    y = np.empty((S, H, dv))
    yvar = np.empty((S, H, dv))
    lib.kla_oracle_decode_step(S, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(a), _ptr(p), _ptr(r),
                               _ptr(lam), _ptr(eta), _ptr(y), _ptr(yvar))
    if per_head:
        yvar = yvar[..., 0].copy()
    if lam_per_slot:
        lam = lam[..., 0].copy()
    return {"y": y, "yvar": yvar, "lam": lam, "eta": eta}


def trace(k, v, a, p, r, lam0=None, eta0=None) -> tuple[np.ndarray, np.ndarray]:
    """Whole (lam, eta) trajectory of one sequence: k, a, p [T, dk]; v, r [T, dv].

    Returns two ``[T+1, dk, dv]`` arrays; row 0 is the prior belief."""
    lib = _load()
    k, v, a, p, r = (_c(x) for x in (k, v, a, p, r))
    T, dk = k.shape
    dv = v.shape[1]
    lam0 = None if lam0 is None else _c(np.broadcast_to(lam0, (dk, dv)))
    eta0 = None if eta0 is None else _c(np.broadcast_to(eta0, (dk, dv)))
    lt = np.empty((T + 1, dk, dv))
    et = np.empty((T + 1, dk, dv))
    lib.kla_oracle_trace(T, dk, dv, _ptr(k), _ptr(v), _ptr(a), _ptr(p), _ptr(r),
                         _ptr(lam0), _ptr(eta0), _ptr(lt), _ptr(et))
    return lt, et


def mobius_matrix(k: float, a: float, p: float, r: float) -> np.ndarray:
    """Per-token 2x2 Moebius matrix of the precision update (Theorem 1)."""
    M = np.empty(4)
    _load().kla_oracle_mobius_matrix(float(k), float(a), float(p), float(r), _ptr(M))
    return M.reshape(2, 2)


def mobius_compose(M2, M1) -> np.ndarray:
    """``M2`` after ``M1`` (Corollary 1)."""
    A, Bm, out = _c(M2).reshape(4), _c(M1).reshape(4), np.empty(4)
    _load().kla_oracle_mobius_compose(_ptr(A), _ptr(Bm), _ptr(out))
    return out.reshape(2, 2)


def mobius_apply(M, lam: float) -> float:
    return float(_load().kla_oracle_mobius_apply(_ptr(_c(M).reshape(4)), float(lam)))


def affine_compose(f2, b2, f1, b1) -> tuple[np.ndarray, np.ndarray]:
    """``(f2, b2)`` after ``(f1, b1)`` for a diagonal gate f over the rows of b (Corollary 2)."""
    b1 = _c(b1)
    b2 = _c(b2)
    shape = np.broadcast_shapes(b1.shape, b2.shape)
    f1 = _c(np.broadcast_to(np.asarray(f1, dtype=np.float64).reshape(
        np.asarray(f1).shape + (1,) * (len(shape) - np.ndim(f1))), shape))
    f2 = _c(np.broadcast_to(np.asarray(f2, dtype=np.float64).reshape(
        np.asarray(f2).shape + (1,) * (len(shape) - np.ndim(f2))), shape))
    b1 = _c(np.broadcast_to(b1, shape))
    b2 = _c(np.broadcast_to(b2, shape))
    fo = np.empty(shape)
    bo = np.empty(shape)
    _load().kla_oracle_affine_compose(int(np.prod(shape)), _ptr(f2), _ptr(b2), _ptr(f1), _ptr(b1),
                                      _ptr(fo), _ptr(bo))
    return fo, bo


# --------------------------------------------------------------------------------------
# OU parameterisation (Sec. 4.1, eq. discretisation; Algorithm 1's OU-Discretisation
# steps): time-invariant parameters a > 0 (mean reversion), p (diffusion scale) and
# delta > 0 (step size), each [H, dk], define the decay and process-noise variance
# shared by every token of every sequence:
#   abar = exp(-a delta),    pbar = p^2 / (2 a) (1 - exp(-2 a delta)).
# The filter is then the one above with abar_t = abar and pbar_t = pbar for all
# (b, t); their gradients are the sums over (b, t) of the per-token ones, taken
# through the discretisation by the chain rule.

def ou_discretise(a, p, delta) -> tuple[np.ndarray, np.ndarray]:
    """Decay abar and process-noise variance pbar of the exactly discretised OU prior."""
    a, p, delta = (_c(x) for x in (a, p, delta))
    abar = np.exp(-a * delta)
    pbar = p * p * (-np.expm1(-2.0 * a * delta)) / (2.0 * a)
    return abar, pbar


def ou_discretise_vjp(a, p, delta, g_abar, g_pbar) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Gradients (da, dp, ddelta) of a loss whose gradients with respect to abar and
    pbar are g_abar and g_pbar (all [H, dk]).

    With E = exp(-2 a delta) = abar^2 and s = (1 - E) / (2 a), so that pbar = p^2 s:
      d abar / d a = -delta abar,   d abar / d delta = -a abar,
      d s / d a = (delta E - s) / a,   d s / d delta = E."""
    a, p, delta, g_abar, g_pbar = (_c(x) for x in (a, p, delta, g_abar, g_pbar))
    abar = np.exp(-a * delta)
    E = abar * abar
    s = -np.expm1(-2.0 * a * delta) / (2.0 * a)
    da = g_abar * (-delta * abar) + g_pbar * p * p * (delta * E - s) / a
    dp = g_pbar * 2.0 * p * s
    ddelta = g_abar * (-a * abar) + g_pbar * p * p * E
    return da, dp, ddelta


def _ou_tokens(a, p, delta, B, T):
    abar, pbar = ou_discretise(a, p, delta)
    shape = (B, T) + abar.shape
    return _c(np.broadcast_to(abar, shape)), _c(np.broadcast_to(pbar, shape))


def forward_ou(q, k, v, a, p, delta, r, lam0=None, eta0=None, nthreads: Optional[int] = None) -> dict:
    """``forward`` with the gates of the OU parameters a, p, delta [H, dk]."""
    B, T = np.shape(k)[:2]
    abar, pbar = _ou_tokens(a, p, delta, B, T)
    return forward(q, k, v, abar, pbar, r, lam0, eta0, nthreads=nthreads)


def backward_ou(q, k, v, a, p, delta, r, lam0, eta0, dy, dlamT=None, detaT=None,
                nthreads: Optional[int] = None, dyvar=None, with_mass: bool = False) -> dict:
    """Gradient of ``forward_ou``: dq, dk, dv, dr, dlam0, deta0 as in ``backward``, and
    da, dp, ddelta [H, dk] for the OU parameters.

    Each parameter gradient is a sum over (b, t) of per-token terms (the gate
    gradients of a token taken through the discretisation).  ``with_mass`` also
    returns ``mass_da``, ``mass_dp``, ``mass_ddelta``: the sum over (b, t) of the
    absolute values of those terms, the scale against which the rounding of such a
    sum is measured (test infrastructure)."""
    B, T = np.shape(k)[:2]
    abar, pbar = _ou_tokens(a, p, delta, B, T)
    out = backward(q, k, v, abar, pbar, r, lam0, eta0, dy, dlamT, detaT, nthreads=nthreads, dyvar=dyvar)
    ga_tok = out.pop("da")
    gp_tok = out.pop("dp")
    g_abar = ga_tok.sum(axis=(0, 1))
    g_pbar = gp_tok.sum(axis=(0, 1))
    out["da"], out["dp"], out["ddelta"] = ou_discretise_vjp(a, p, delta, g_abar, g_pbar)
    if with_mass:
        for name, (ca, cp) in zip(("mass_da", "mass_dp", "mass_ddelta"),
                                  zip(*(ou_discretise_vjp(a, p, delta, np.ones_like(g_abar) * (i == 0),
                                                          np.ones_like(g_pbar) * (i == 1)) for i in (0, 1)))):
            out[name] = np.abs(ga_tok * ca + gp_tok * cp).sum(axis=(0, 1))
    return out


def decode_step_ou(q, k, v, a, p, delta, r, lam, eta) -> dict:
    """``decode_step`` with the gates of the OU parameters a, p, delta [H, dk]."""
    abar, pbar = ou_discretise(a, p, delta)
    S = np.shape(k)[0]
    shape = (S,) + abar.shape
    return decode_step(q, k, v, np.broadcast_to(abar, shape), np.broadcast_to(pbar, shape), r, lam, eta)


# --------------------------------------------------------------------------------------
# Gates per (key slot, value channel): Algorithm 1 gives A, P, Delta (and so abar, pbar)
# the shape (N, D), time-invariant, per head: [H, dk, dv].  With the observation
# precision per value channel (r [B, T, H, dv]) every element (n, d) of a head is its
# own scalar filter with its own gates.

def forward_nd(q, k, v, abar, pbar, r, lam0=None, eta0=None, nthreads: Optional[int] = None) -> dict:
    """The filter with gates abar, pbar [H, dk, dv] (the same for every token); r [B, T, H, dv].
    Returns y, yvar [B, T, H, dv], lamT, etaT [B, H, dk, dv]."""
    lib = _load()
    q, k, v, r, abar, pbar = (_c(x) for x in (q, k, v, r, abar, pbar))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    lam0 = None if lam0 is None else _c(lam0)
    eta0 = None if eta0 is None else _c(eta0)
    y = np.empty((B, T, H, dv))
    yvar = np.empty((B, T, H, dv))
    lamT = np.empty((B, H, dk, dv))
    etaT = np.empty((B, H, dk, dv))
    lib.kla_oracle_forward_nd(B, T, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(abar), _ptr(pbar), _ptr(r),
                              _ptr(lam0), _ptr(eta0), _ptr(y), _ptr(yvar), _ptr(lamT), _ptr(etaT),
                              nthreads or default_threads())
    return {"y": y, "yvar": yvar, "lamT": lamT, "etaT": etaT}


def backward_nd(q, k, v, abar, pbar, r, lam0, eta0, dy, dlamT=None, detaT=None, dyvar=None,
                coef=None, nthreads: Optional[int] = None) -> dict:
    """Gradient of ``forward_nd``: dq, dk [B, T, H, dk], dv, dr [B, T, H, dv], dlam0, deta0
    [B, H, dk, dv], and the gate gradients g_abar, g_pbar [H, dk, dv] (sums over (b, t)).
    ``coef`` = (ca, cp), each [3, H, dk, dv]: also return ``mass`` [3, H, dk, dv], the sums
    over (b, t) of |ca[j] dabar_t + cp[j] dpbar_t|."""
    lib = _load()
    q, k, v, r, abar, pbar, dy = (_c(x) for x in (q, k, v, r, abar, pbar, dy))
    B, T, H, dk = k.shape
    dv = v.shape[-1]
    lam0, eta0, dlamT, detaT, dyvar = (None if x is None else _c(x) for x in (lam0, eta0, dlamT, detaT, dyvar))
    ca, cp = (np.zeros((3, H, dk, dv)), np.zeros((3, H, dk, dv))) if coef is None else (_c(coef[0]), _c(coef[1]))
    out = {"dq": np.empty((B, T, H, dk)), "dk": np.empty((B, T, H, dk)), "dv": np.empty((B, T, H, dv)),
           "dr": np.empty((B, T, H, dv)), "dlam0": np.empty((B, H, dk, dv)), "deta0": np.empty((B, H, dk, dv))}
    ga = np.empty((B, H, dk, dv))
    gp = np.empty((B, H, dk, dv))
    mass = np.empty((3, B, H, dk, dv))
    lib.kla_oracle_backward_nd(B, T, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(abar), _ptr(pbar), _ptr(r),
                               _ptr(lam0), _ptr(eta0), _ptr(dy), _ptr(dyvar), _ptr(dlamT), _ptr(detaT),
                               _ptr(out["dq"]), _ptr(out["dk"]), _ptr(out["dv"]), _ptr(out["dr"]),
                               _ptr(out["dlam0"]), _ptr(out["deta0"]), _ptr(ca), _ptr(cp), _ptr(ga), _ptr(gp),
                               _ptr(mass), nthreads or default_threads())
    out["g_abar"] = ga.sum(axis=0)
    out["g_pbar"] = gp.sum(axis=0)
    if coef is not None:
        out["mass"] = mass.sum(axis=1)
    return out


def forward_ou_nd(q, k, v, a, p, delta, r, lam0=None, eta0=None, nthreads: Optional[int] = None) -> dict:
    """``forward_nd`` with the gates of OU parameters a, p, delta [H, dk, dv]."""
    abar, pbar = ou_discretise(a, p, delta)
    return forward_nd(q, k, v, abar, pbar, r, lam0, eta0, nthreads=nthreads)


def backward_ou_nd(q, k, v, a, p, delta, r, lam0, eta0, dy, dlamT=None, detaT=None, dyvar=None,
                   nthreads: Optional[int] = None) -> dict:
    """Gradient of ``forward_ou_nd``: as ``backward_nd`` for the per-token tensors and the
    initial belief, and da, dp, ddelta [H, dk, dv] with the masses mass_da, mass_dp,
    mass_ddelta of their terms (sums over (b, t) of the absolute per-token terms)."""
    a, p, delta = (_c(x) for x in (a, p, delta))
    abar, pbar = ou_discretise(a, p, delta)
    one, zero = np.ones_like(a), np.zeros_like(a)
    ca = np.stack(ou_discretise_vjp(a, p, delta, one, zero))    # d(da, dp, ddelta) / d g_abar
    cp = np.stack(ou_discretise_vjp(a, p, delta, zero, one))    # ... / d g_pbar
    out = backward_nd(q, k, v, abar, pbar, r, lam0, eta0, dy, dlamT, detaT, dyvar, coef=(ca, cp),
                      nthreads=nthreads)
    ga, gp = out.pop("g_abar"), out.pop("g_pbar")
    out["da"], out["dp"], out["ddelta"] = ou_discretise_vjp(a, p, delta, ga, gp)
    m = out.pop("mass")
    out["mass_da"], out["mass_dp"], out["mass_ddelta"] = m[0], m[1], m[2]
    return out
