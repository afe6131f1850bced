"""fp64 oracle of the scaffolding around the KLA layer (TEST INFRASTRUCTURE ONLY).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
use this module; it shares no code with the GPU kernels.

The paper's block (Sec. 4.4 and the architecture paragraph of Appendix A)
follows Mamba: a causal depthwise 1D convolution of kernel size 4 with a SiLU
activation, QK-norm on the query and key, and an elementwise gate.  The paper
fixes none of their details; the readings used here:

* conv: ``u[b, t, c] = silu(bias[c] + sum_j w[c, j] x[b, t - 3 + j, c])`` with
  ``x`` zero before the first token (tap ``j = 3`` is the current token);
* QK-norm: RMS normalisation of each row (one head's q or k of one token) with
  a learnable weight shared by the rows, ``out = x / sqrt(mean(x^2) + eps) * w``;
* gate: ``out = y * silu(z)``.

Each forward is the definition written out; each backward is its derivative
taken by hand (pinned by finite differences in the tests).
"""
from __future__ import annotations

import numpy as np

KCONV = 4


def _c(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def silu(x):
    return x * sigmoid(x)


def silu_grad(x):
    """d silu / dx = s (1 + x (1 - s)), s = sigmoid(x)."""
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def conv_preact(x, w, bias=None):
    """``bias[c] + sum_j w[c, j] x[b, t - 3 + j, c]`` for x [B, T, C], w [C, 4]."""
    x, w = _c(x), _c(w)
    B, T, C = x.shape
    out = np.zeros((B, T, C)) if bias is None else np.broadcast_to(_c(bias), (B, T, C)).copy()
    for j in range(KCONV):
        lag = KCONV - 1 - j          # tap j looks lag tokens back
        if lag >= T:
            continue
        out[:, lag:, :] += w[:, j] * x[:, :T - lag, :]
    return out


def conv_silu_forward(x, w, bias=None):
    return silu(conv_preact(x, w, bias))


def conv_silu_backward(x, w, bias, du):
    """(dx, dw, dbias) of ``conv_silu_forward`` for the upstream gradient du."""
    x, w, du = _c(x), _c(w), _c(du)
    B, T, C = x.shape
    ds = du * silu_grad(conv_preact(x, w, bias))
    dx = np.zeros_like(x)
    dw = np.zeros_like(w)
    for j in range(KCONV):
        lag = KCONV - 1 - j
        if lag >= T:
            continue
        dx[:, :T - lag, :] += w[:, j] * ds[:, lag:, :]
        dw[:, j] = (ds[:, lag:, :] * x[:, :T - lag, :]).sum(axis=(0, 1))
    return dx, dw, ds.sum(axis=(0, 1))


def rmsnorm_forward(x, w, eps):
    """Rows of x [..., n]: x / sqrt(mean(x^2) + eps) * w; also returns 1 / rms per row."""
    x, w = _c(x), _c(w)
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * rstd * w, rstd[..., 0]


def rmsnorm_backward(x, w, eps, dout):
    """(dx, dw): with xh = x rstd, dx = rstd (w dout - xh mean(xh w dout)), dw = sum over rows of dout xh."""
    x, w, dout = _c(x), _c(w), _c(dout)
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    xh = x * rstd
    g = w * dout
    dx = rstd * (g - xh * np.mean(xh * g, axis=-1, keepdims=True))
    dw = (dout * xh).reshape(-1, x.shape[-1]).sum(axis=0)
    return dx, dw


def gate_forward(y, z):
    return _c(y) * silu(_c(z))


def gate_backward(y, z, dout):
    y, z, dout = _c(y), _c(z), _c(dout)
    return dout * silu(z), dout * y * silu_grad(z)
