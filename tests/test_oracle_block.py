"""Pins of the block-scaffolding oracle (oracle/block.py): causal conv + SiLU,
QK-norm (RMS normalisation), gate.

* the convolution against numpy's full discrete convolution per channel;
* SiLU against its definition and its derivative against central differences;
* RMS normalisation: unit mean square with a unit weight and eps = 0, and
  invariance under scaling of a row;
* every backward against central differences of its forward;
* planted mistakes in a copy of the module fail these pins.
"""
import importlib.util
import os

import numpy as np
import pytest

from oracle import block as OB

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _fd(f, x, h=1e-6):
    g = np.zeros_like(x)
    for i in np.ndindex(x.shape):
        old = x[i]
        x[i] = old + h
        fp = f()
        x[i] = old - h
        fm = f()
        x[i] = old
        g[i] = (fp - fm) / (2 * h)
    return g


def _conv_battery(ob) -> bool:
    g = np.random.default_rng(0)
    B, T, C = 2, 9, 3
    x = g.standard_normal((B, T, C))
    w = g.standard_normal((C, 4))
    bias = g.standard_normal(C)
    pre = ob.conv_preact(x, w, bias)
    ok = True
    for b in range(B):
        for c in range(C):
            ref = np.convolve(x[b, :, c], w[c, ::-1])[:T] + bias[c]
            ok &= np.allclose(pre[b, :, c], ref, rtol=1e-13, atol=1e-13)
    ok &= np.allclose(ob.conv_silu_forward(x, w, bias), pre / (1 + np.exp(-pre)), rtol=1e-13)
    return bool(ok)


def _grad_battery(ob) -> bool:
    g = np.random.default_rng(1)
    ok = True
    # conv + SiLU
    B, T, C = 2, 6, 3
    x = g.standard_normal((B, T, C))
    w = g.standard_normal((C, 4))
    bias = g.standard_normal(C)
    du = g.standard_normal((B, T, C))
    dx, dw, db = ob.conv_silu_backward(x, w, bias, du)
    loss = lambda: float((ob.conv_silu_forward(x, w, bias) * du).sum())
    ok &= np.allclose(dx, _fd(loss, x), rtol=1e-6, atol=1e-8)
    ok &= np.allclose(dw, _fd(loss, w), rtol=1e-6, atol=1e-8)
    ok &= np.allclose(db, _fd(loss, bias), rtol=1e-6, atol=1e-8)
    # RMS normalisation
    xr = g.standard_normal((5, 8))
    wr = g.standard_normal(8)
    dout = g.standard_normal((5, 8))
    dxr, dwr = ob.rmsnorm_backward(xr, wr, 1e-3, dout)
    loss = lambda: float((ob.rmsnorm_forward(xr, wr, 1e-3)[0] * dout).sum())
    ok &= np.allclose(dxr, _fd(loss, xr), rtol=1e-6, atol=1e-8)
    ok &= np.allclose(dwr, _fd(loss, wr), rtol=1e-6, atol=1e-8)
    # gate
    y = g.standard_normal((4, 7))
    z = g.standard_normal((4, 7))
    do = g.standard_normal((4, 7))
    dy, dz = ob.gate_backward(y, z, do)
    loss = lambda: float((ob.gate_forward(y, z) * do).sum())
    ok &= np.allclose(dy, _fd(loss, y), rtol=1e-6, atol=1e-8)
    ok &= np.allclose(dz, _fd(loss, z), rtol=1e-6, atol=1e-8)
    return bool(ok)


def test_conv_matches_numpy_convolution():
    assert _conv_battery(OB)


def test_backwards_match_central_differences():
    assert _grad_battery(OB)


def test_silu_definition_and_derivative():
    x = np.linspace(-6, 6, 25)
    np.testing.assert_allclose(OB.silu(x), x / (1 + np.exp(-x)), rtol=1e-14)
    h = 1e-6
    np.testing.assert_allclose(OB.silu_grad(x), (OB.silu(x + h) - OB.silu(x - h)) / (2 * h), rtol=1e-7, atol=1e-9)


def test_rmsnorm_unit_mean_square_and_scale_invariance():
    g = np.random.default_rng(2)
    x = g.standard_normal((6, 16))
    out, rstd = OB.rmsnorm_forward(x, np.ones(16), 0.0)
    np.testing.assert_allclose(np.mean(out * out, axis=-1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(rstd, 1.0 / np.sqrt(np.mean(x * x, axis=-1)), rtol=1e-14)
    out2, _ = OB.rmsnorm_forward(37.5 * x, np.ones(16), 0.0)
    np.testing.assert_allclose(out2, out, rtol=1e-13)


def test_conv_shorter_than_kernel():
    g = np.random.default_rng(3)
    x = g.standard_normal((1, 2, 2))
    w = g.standard_normal((2, 4))
    pre = OB.conv_preact(x, w)
    np.testing.assert_allclose(pre[0, 0], w[:, 3] * x[0, 0], rtol=1e-14)
    np.testing.assert_allclose(pre[0, 1], w[:, 3] * x[0, 1] + w[:, 2] * x[0, 0], rtol=1e-14)


BLOCK_MUTATIONS = {
    "conv_taps_reversed": ("lag = KCONV - 1 - j          # tap j looks lag tokens back",
                           "lag = j"),
    "silu_grad_missing_term": ("return s * (1.0 + x * (1.0 - s))", "return s * (1.0 + x * s)"),
    "rmsnorm_dx_missing_projection": ("dx = rstd * (g - xh * np.mean(xh * g, axis=-1, keepdims=True))",
                                      "dx = rstd * g"),
    "gate_dz_without_y": ("return dout * silu(z), dout * y * silu_grad(z)",
                          "return dout * silu(z), dout * silu_grad(z)"),
}


@pytest.mark.parametrize("name", sorted(BLOCK_MUTATIONS))
def test_planted_block_mistake_is_caught(tmp_path, name):
    old, new = BLOCK_MUTATIONS[name]
    src = open(os.path.join(ROOT, "oracle", "block.py")).read()
    assert src.count(old) == 1, old
    path = tmp_path / "block_mut.py"
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"block_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert not (_conv_battery(mod) and _grad_battery(mod)), f"mutation {name} passed the pins"
