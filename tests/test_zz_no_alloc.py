"""The allocation-free backward (kla_backward_noalloc, the library's per-GPU static
workspace) against kla_backward with a caller workspace: the same kernels, so the
results must agree bit for bit.  Two calls in a row, the second on a smaller problem
(the static workspace keeps the first call's contents)."""
import ctypes

import numpy as np
import pytest

import kla_inputs as K
from kla_testutil import log, to_torch

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
GRADS = ("dq", "dk", "dv", "da", "dp", "dr", "dlam0", "deta0")


@pytest.fixture(scope="module")
def kla():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2602_10743_amd as lib
    lib._load()
    return lib


def _one(kla, B, T, H, dk, dv, dtype, dist, seed):
    case = K.random_case(B, T, H, dk, dv, dtype, seed=seed, dist=dist)
    x = {n: to_torch(case[n], dtype, DEV) for n in K.NAMES + ("dy",)}
    g = np.random.default_rng(seed)
    f32 = lambda a: torch.tensor(a.astype(np.float32), device=DEV)
    lam0, eta0 = f32(0.5 + g.random((B, H, dk))), f32(g.standard_normal((B, H, dk, dv)))
    dlamT, detaT = f32(g.standard_normal((B, H, dk))), f32(g.standard_normal((B, H, dk, dv)))
    dyvar = f32(g.standard_normal((B, T, H)))
    saved = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], lam0, eta0, save=True)["saved"]
    args = (x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], lam0, eta0, x["dy"], dlamT, detaT)
    ref = kla.kla_backward(*args, saved=saved, dyvar=dyvar)
    got = kla.kla_backward_noalloc(*args, saved=saved, dyvar=dyvar)
    torch.cuda.synchronize()
    for n in GRADS:
        assert torch.equal(got[n], ref[n]), f"{n} differs from kla_backward (B{B} T{T} H{H} d{dk}/{dv} {dtype})"


# bf16 at these shapes runs the chunked kernels; fp32 the token-recurrent ones (d128, 64/32)
# and the chunked fp64 ones (32/32, 32/16)
@pytest.mark.parametrize("dtype,first,second", [
    ("bf16", (2, 300, 4, 128, 128), (1, 70, 2, 64, 32)),
    ("f32", (2, 300, 4, 128, 128), (1, 70, 2, 64, 32)),
    ("f32", (2, 300, 4, 32, 32), (1, 45, 2, 32, 16)),
])
def test_noalloc_matches_backward_twice(kla, dtype, first, second):
    log(f"noalloc {dtype}: B T H dk dv {first}, then {second}")
    _one(kla, *first, dtype, "lm", seed=11)
    _one(kla, *second, dtype, "lm", seed=12)


def test_noalloc_rejects_oversize_and_missing_context(kla):
    lib = kla._load()
    fake = ctypes.c_void_p(0x10000)   # aligned, never dereferenced: the call returns first
    big = kla._Desc(64, 4096, 8, 128, 128, 1)      # dr parts of 64 MiB + the flag: over the limit
    ptrs = [fake] * 6 + [None, None, fake, fake, None, None, None] + [fake] * 6 + [None, None]
    assert lib.kla_backward_noalloc(ctypes.byref(big), *ptrs, None) == 5      # KLA_ERR_WORKSPACE
    small = kla._Desc(1, 8, 1, 32, 32, 1)
    no_ctx = list(ptrs)
    no_ctx[8] = None
    assert lib.kla_backward_noalloc(ctypes.byref(small), *no_ctx, None) == 1  # KLA_ERR_NULL
