"""Host-side checks of the C ABI (no GPU work): the library loads, exports every
symbol include/kla.h declares, and rejects bad arguments before launching."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kla.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kla_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2602_10743_amd as K
    return K._load()


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("kla_forward", "kla_backward", "kla_decode_step", "kla_status_string",
              "kla_forward_workspace", "kla_backward_workspace", "kla_saved_bytes"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), f"{name} declared in kla.h but not exported"


def test_status_strings(lib):
    import paper_2602_10743_amd as K
    for code in range(8):
        assert K.kla_status_string(code).startswith("KLA_")


def _desc(B=1, T=8, H=1, dk=16, dv=16, dtype=0):
    import paper_2602_10743_amd as K
    return K._Desc(B, T, H, dk, dv, dtype)


def test_workspace_queries(lib):
    import paper_2602_10743_amd as K
    assert K.kla_forward_workspace(_desc()) > 0
    assert K.kla_backward_workspace(_desc(), False) > 0
    assert K.kla_forward_workspace(_desc(dk=24)) == 0          # unsupported width
    assert K.kla_backward_workspace(_desc(dtype=7), True) == 0  # unknown dtype


def _fwd(lib, desc, ptrs, ws_bytes=256):
    return lib.kla_forward(ctypes.byref(desc), *ptrs, ws_bytes, None)


def test_forward_argument_errors(lib):
    fake = ctypes.c_void_p(0x10000)       # aligned, never dereferenced: the call returns first
    odd = ctypes.c_void_p(0x10004)
    ok = [fake] * 6 + [None, None, fake, None, None, None, None, fake]
    assert _fwd(lib, _desc(dk=24), ok) == 2                        # KLA_ERR_SHAPE
    assert _fwd(lib, _desc(dtype=5), ok) == 3                      # KLA_ERR_DTYPE
    assert _fwd(lib, _desc(B=0), ok) == 2
    assert _fwd(lib, _desc(T=-1), ok) == 2
    assert lib.kla_forward(None, *ok, 256, None) == 1              # KLA_ERR_NULL
    bad = list(ok)
    bad[0] = None
    assert _fwd(lib, _desc(), bad) == 1
    bad = list(ok)
    bad[2] = odd
    assert _fwd(lib, _desc(), bad) == 4                            # KLA_ERR_ALIGN
    assert _fwd(lib, _desc(), ok, ws_bytes=0) == 5                 # KLA_ERR_WORKSPACE
    bad = list(ok)
    bad[13] = None
    assert _fwd(lib, _desc(), bad) == 5


def test_backward_and_decode_argument_errors(lib):
    fake = ctypes.c_void_p(0x10000)
    d = _desc()
    # q k v a p r lam0 eta0 saved dy dyvar dlamT detaT dq dk dv da dp dr dlam0 deta0 ws
    args = [fake] * 6 + [None, None, None] + [fake, None, None, None] + [fake] * 6 + [None, None] + [fake]
    assert lib.kla_backward(ctypes.byref(d), *args, 0, None) == 5
    bad = list(args)
    bad[9] = None                                                  # dy
    assert lib.kla_backward(ctypes.byref(d), *bad, 1 << 40, None) == 1
    dec = [fake] * 6 + [fake, fake, fake, None, None]
    assert lib.kla_decode_step(4, 2, 16, 48, 0, *dec) == 2
    assert lib.kla_decode_step(4, 2, 16, 16, 9, *dec) == 3
    bad = list(dec)
    bad[6] = None
    assert lib.kla_decode_step(4, 2, 16, 16, 0, *bad) == 1


def test_binding_refuses_cpu_tensors():
    import torch
    import paper_2602_10743_amd as K
    x = torch.zeros(1, 4, 1, 16)
    with pytest.raises(ValueError, match="GPU"):
        K.kla_forward(x, x, x, x, x, torch.zeros(1, 4, 1))


def test_ou_entry_points_declared_and_sized(lib):
    import paper_2602_10743_amd as K
    names = _declared()
    for n in ("kla_forward_ou", "kla_backward_ou", "kla_decode_step_ou", "kla_backward_ou_workspace"):
        assert n in names
    for d in (_desc(), _desc(B=3, T=70, H=2, dk=64, dv=32, dtype=1)):
        # the OU backward adds the per-part gate-gradient sums to the plain workspace
        for saved in (False, True):
            assert K.kla_backward_ou_workspace(d, saved) > K.kla_backward_workspace(d, saved)
    assert K.kla_backward_ou_workspace(_desc(dk=24), False) == 0


def test_ou_argument_errors(lib):
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10004)
    d = _desc()
    # q k v a p delta r lam0 eta0 y yvar lamT etaT saved ws
    ok = [fake] * 7 + [None, None, fake, None, None, None, None, fake]
    assert lib.kla_forward_ou(ctypes.byref(_desc(dk=24)), *ok, 256, None) == 2
    for i in (3, 4, 5):                                            # a, p, delta
        bad = list(ok)
        bad[i] = None
        assert lib.kla_forward_ou(ctypes.byref(d), *bad, 256, None) == 1
    bad = list(ok)
    bad[5] = odd
    assert lib.kla_forward_ou(ctypes.byref(d), *bad, 256, None) == 4
    assert lib.kla_forward_ou(ctypes.byref(d), *ok, 0, None) == 5
    # q k v a p delta r lam0 eta0 saved dy dyvar dlamT detaT dq dk dv da dp ddelta dr dlam0 deta0 ws
    bwd = [fake] * 7 + [None, None, None] + [fake, None, None, None] + [fake] * 7 + [None, None] + [fake]
    assert lib.kla_backward_ou(ctypes.byref(d), *bwd, 0, None) == 5
    for i in (17, 18, 19):                                         # da, dp, ddelta
        bad = list(bwd)
        bad[i] = None
        assert lib.kla_backward_ou(ctypes.byref(d), *bad, 1 << 40, None) == 1
    dec = [fake] * 7 + [fake, fake, fake, None, None]
    assert lib.kla_decode_step_ou(4, 2, 16, 48, 0, *dec) == 2
    bad = list(dec)
    bad[5] = None
    assert lib.kla_decode_step_ou(4, 2, 16, 16, 0, *bad) == 1


def test_per_channel_entry_points(lib):
    import paper_2602_10743_amd as K
    names = _declared()
    for n in ("kla_forward_pc", "kla_backward_pc", "kla_decode_step_pc", "kla_saved_pc_bytes",
              "kla_backward_pc_workspace"):
        assert n in names
    d = _desc(B=2, T=20, H=3, dk=32, dv=16)
    # the saved context holds lam and eta at every 8th token: 3 checkpoints of [B, H, dk, dv],
    # in the arithmetic type (fp64 for fp32 inputs, fp32 for bf16 inputs)
    assert lib.kla_saved_pc_bytes(ctypes.byref(d)) == 2 * 2 * 3 * 3 * 32 * 16 * 8
    assert lib.kla_saved_pc_bytes(ctypes.byref(_desc(B=2, T=20, H=3, dk=32, dv=16, dtype=1))) == \
        2 * 2 * 3 * 3 * 32 * 16 * 4
    assert lib.kla_backward_pc_workspace(ctypes.byref(d), 0) > lib.kla_backward_pc_workspace(ctypes.byref(d), 1)
    fake = ctypes.c_void_p(0x10000)
    # q k v a p r lam0 eta0 y yvar lamT etaT saved ws
    fwd = [fake] * 6 + [None, None, fake, None, None, None, None, fake]
    assert lib.kla_forward_pc(ctypes.byref(_desc(dk=24)), *fwd, 256, None) == 2
    bad = list(fwd)
    bad[5] = None                                                  # r
    assert lib.kla_forward_pc(ctypes.byref(d), *bad, 256, None) == 1
    assert lib.kla_forward_pc(ctypes.byref(d), *fwd, 0, None) == 5
    # q k v a p r lam0 eta0 saved dy dyvar dlamT detaT dq dk dv da dp dr dlam0 deta0 ws
    bwd = [fake] * 6 + [None, None, None] + [fake, None, None, None] + [fake] * 6 + [None, None] + [fake]
    assert lib.kla_backward_pc(ctypes.byref(d), *bwd, 0, None) == 5
    bad = list(bwd)
    bad[18] = None                                                 # dr
    assert lib.kla_backward_pc(ctypes.byref(d), *bad, 1 << 40, None) == 1


def test_block_scaffolding_entry_points(lib):
    names = _declared()
    for n in ("kla_conv_silu_forward", "kla_conv_silu_backward", "kla_conv_silu_workspace", "kla_qk_norm_forward",
              "kla_qk_norm_backward", "kla_qk_norm_workspace", "kla_gate_forward", "kla_gate_backward"):
        assert n in names
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10004)
    assert lib.kla_conv_silu_forward(2, 10, 12, 1, fake, fake, None, fake, None) == 2    # C % 8 for bf16
    assert lib.kla_conv_silu_forward(2, 10, 16, 3, fake, fake, None, fake, None) == 3    # dtype
    assert lib.kla_conv_silu_forward(2, 10, 16, 1, None, fake, None, fake, None) == 1    # x
    assert lib.kla_conv_silu_forward(2, 10, 16, 1, odd, fake, None, fake, None) == 4     # alignment
    assert lib.kla_conv_silu_backward(2, 10, 16, 1, fake, fake, None, fake, fake, fake, None, fake, 0, None) == 5
    assert lib.kla_conv_silu_workspace(2, 130, 16) == 2 * 3 * 16 * 5 * 4   # one part per 64 tokens
    assert lib.kla_qk_norm_forward(10, 24, 1, fake, fake, ctypes.c_float(1e-6), fake, None, None) == 2
    assert lib.kla_qk_norm_forward(10, 32, 1, fake, None, ctypes.c_float(1e-6), fake, None, None) == 1
    assert lib.kla_qk_norm_backward(10, 32, 1, fake, fake, fake, fake, fake, fake, fake, 0, None) == 5
    assert lib.kla_gate_forward(12, 1, fake, fake, fake, None) == 2                       # n % 8 for bf16
    assert lib.kla_gate_backward(16, 1, fake, fake, None, fake, fake, None) == 1


def test_saved_context_layout_follows_the_backward(lib):
    """The forward fills the saved context in the layout of the backward that will read
    it: bf16 with dk >= 32 but dv = 16 runs the token-recurrent backward, so its context
    is the per-token precision plus a state checkpoint every 64 tokens, not the chunked one."""
    import paper_2602_10743_amd as K
    B, T, H, dk = 2, 64, 3, 64
    nck = (T + 63) // 64
    rec = (B * T * H * dk + B * H * nck * dk * 16) * 4   # bf16 inputs: fp32 arithmetic
    assert K.kla_saved_bytes(_desc(B, T, H, dk, 16, 1)) == rec
    nchunk = (T + 31) // 32
    chunked = B * H * dk * (3 * nchunk + (nchunk + 1) * 32) * 4   # walk state (3 rows), then states
    assert K.kla_saved_bytes(_desc(B, T, H, dk, 32, 1)) == chunked
    # fp32 inputs: the chunked fp64 path at dk, dv <= 32 (lam at every chunk start, then the
    # states, fp64), the token-recurrent fp64 kernels above
    for dk2, dv2 in ((32, 32), (32, 16), (16, 32), (16, 16)):
        c64 = B * H * dk2 * (nchunk + (nchunk + 1) * dv2) * 8
        assert K.kla_saved_bytes(_desc(B, T, H, dk2, dv2, 0)) == c64
        # with a saved context the fp64 chunk backward needs only the validation flag's slot;
        # without one, room for the recomputed context and a scratch output
        with_ctx = K.kla_backward_workspace(_desc(B, T, H, dk2, dv2, 0), True)
        assert 0 < with_ctx <= 256
        assert K.kla_backward_workspace(_desc(B, T, H, dk2, dv2, 0), False) >= with_ctx + c64 + B * T * H * dv2 * 4
    rec64 = (B * T * H * 64 + B * H * nck * 64 * 32) * 8
    assert K.kla_saved_bytes(_desc(B, T, H, 64, 32, 0)) == rec64
