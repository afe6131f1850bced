"""Kalman Linear Attention filter layer on MI355X (gfx950): Python binding.

A thin ctypes binding over ``libkla.so`` whose functions carry the names of the
C ABI in ``include/kla.h``.  It only marshals arguments: it checks shapes and
dtypes, allocates outputs and workspace through torch (device memory and
streams are all torch is used for) and passes raw device pointers and the
current HIP stream to the library, where every step of the filter runs.

There is no fallback: if the HIP library is missing or the tensors are not on
a GPU, every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = ["kla_forward", "kla_backward", "kla_backward_noalloc", "kla_decode_step", "kla_status_string",
           "kla_forward_workspace", "kla_backward_workspace", "kla_saved_bytes",
           "kla_forward_ou", "kla_backward_ou", "kla_decode_step_ou", "kla_backward_ou_workspace",
           "kla_forward_pc", "kla_backward_pc", "kla_decode_step_pc",
           "kla_forward_pc_ou", "kla_backward_pc_ou", "kla_decode_step_pc_ou", "KLAFilterPcOU", "kla_filter_pc_ou",
           "kla_conv_silu_forward", "kla_conv_silu_backward", "kla_qk_norm_forward", "kla_qk_norm_backward",
           "kla_gate_forward", "kla_gate_backward",
           "kla_mc_sample", "kla_mc_sample_backward", "kla_mc_nll", "kla_mc_nll_backward", "KLAMCSample",
           "KLAMCNLL", "kla_mc_nll_loss",
           "KLAError", "KLAFilter", "kla_filter", "KLAFilterOU", "kla_filter_ou", "library_path"]

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libkla.so")

KLA_F32, KLA_BF16 = 0, 1
_DTYPES = {torch.float32: KLA_F32, torch.bfloat16: KLA_BF16}


class KLAError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {kla_status_string(status)} (status {status})")


class _Desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("dk", ctypes.c_int32), ("dv", ctypes.c_int32), ("dtype", ctypes.c_int32)]


_lib = None
_VP = ctypes.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(library_path):
        raise ImportError(f"KLA HIP library not built: {library_path} is missing "
                          "(build it with `python paper_2602_10743_amd/build.py`)")
    lib = ctypes.CDLL(library_path)
    D = ctypes.POINTER(_Desc)
    lib.kla_forward_workspace.argtypes = [D]
    lib.kla_forward_workspace.restype = ctypes.c_size_t
    lib.kla_saved_bytes.argtypes = [D]
    lib.kla_saved_bytes.restype = ctypes.c_size_t
    lib.kla_backward_workspace.argtypes = [D, ctypes.c_int]
    lib.kla_backward_workspace.restype = ctypes.c_size_t
    lib.kla_forward.argtypes = [D] + [_VP] * 14 + [ctypes.c_size_t, _VP]
    lib.kla_forward.restype = ctypes.c_int
    lib.kla_backward.argtypes = [D] + [_VP] * 22 + [ctypes.c_size_t, _VP]
    lib.kla_backward.restype = ctypes.c_int
    lib.kla_backward_noalloc.argtypes = [D] + [_VP] * 22
    lib.kla_backward_noalloc.restype = ctypes.c_int
    lib.kla_decode_step.argtypes = [ctypes.c_int32] * 5 + [_VP] * 11
    lib.kla_decode_step.restype = ctypes.c_int
    lib.kla_backward_ou_workspace.argtypes = [D, ctypes.c_int]
    lib.kla_backward_ou_workspace.restype = ctypes.c_size_t
    lib.kla_forward_ou.argtypes = [D] + [_VP] * 15 + [ctypes.c_size_t, _VP]
    lib.kla_forward_ou.restype = ctypes.c_int
    lib.kla_backward_ou.argtypes = [D] + [_VP] * 24 + [ctypes.c_size_t, _VP]
    lib.kla_backward_ou.restype = ctypes.c_int
    lib.kla_decode_step_ou.argtypes = [ctypes.c_int32] * 5 + [_VP] * 12
    lib.kla_decode_step_ou.restype = ctypes.c_int
    lib.kla_forward_pc.argtypes = [D] + [_VP] * 14 + [ctypes.c_size_t, _VP]
    lib.kla_forward_pc.restype = ctypes.c_int
    lib.kla_backward_pc.argtypes = [D] + [_VP] * 22 + [ctypes.c_size_t, _VP]
    lib.kla_backward_pc.restype = ctypes.c_int
    lib.kla_saved_pc_bytes.argtypes = [D]
    lib.kla_saved_pc_bytes.restype = ctypes.c_size_t
    lib.kla_backward_pc_workspace.argtypes = [D, ctypes.c_int]
    lib.kla_backward_pc_workspace.restype = ctypes.c_size_t
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.kla_conv_silu_workspace.argtypes = [i32] * 3
    lib.kla_conv_silu_workspace.restype = ctypes.c_size_t
    lib.kla_conv_silu_forward.argtypes = [i32] * 4 + [_VP] * 5
    lib.kla_conv_silu_backward.argtypes = [i32] * 4 + [_VP] * 8 + [ctypes.c_size_t, _VP]
    lib.kla_qk_norm_workspace.argtypes = [i32]
    lib.kla_qk_norm_workspace.restype = ctypes.c_size_t
    lib.kla_qk_norm_forward.argtypes = [i64, i32, i32, _VP, _VP, ctypes.c_float, _VP, _VP, _VP]
    lib.kla_qk_norm_backward.argtypes = [i64, i32, i32] + [_VP] * 7 + [ctypes.c_size_t, _VP]
    lib.kla_gate_forward.argtypes = [i64, i32] + [_VP] * 4
    lib.kla_gate_backward.argtypes = [i64, i32] + [_VP] * 6
    for fn in ("kla_conv_silu_forward", "kla_conv_silu_backward", "kla_qk_norm_forward", "kla_qk_norm_backward",
               "kla_gate_forward", "kla_gate_backward"):
        getattr(lib, fn).restype = ctypes.c_int
    lib.kla_backward_pc_ou_workspace.argtypes = [D, ctypes.c_int]
    lib.kla_backward_pc_ou_workspace.restype = ctypes.c_size_t
    lib.kla_forward_pc_ou.argtypes = [D] + [_VP] * 15 + [ctypes.c_size_t, _VP]
    lib.kla_forward_pc_ou.restype = ctypes.c_int
    lib.kla_backward_pc_ou.argtypes = [D] + [_VP] * 24 + [ctypes.c_size_t, _VP]
    lib.kla_backward_pc_ou.restype = ctypes.c_int
    lib.kla_decode_step_pc_ou.argtypes = [ctypes.c_int32] * 5 + [_VP] * 12
    lib.kla_decode_step_pc_ou.restype = ctypes.c_int
    lib.kla_decode_step_pc.argtypes = [ctypes.c_int32] * 5 + [_VP] * 11
    lib.kla_decode_step_pc.restype = ctypes.c_int
    u64 = ctypes.c_uint64
    lib.kla_mc_sample.argtypes = [i32] * 6 + [u64] + [_VP] * 4
    lib.kla_mc_sample_backward.argtypes = [i32] * 6 + [u64] + [_VP] * 5
    lib.kla_mc_nll.argtypes = [i32, i64] + [_VP] * 3
    lib.kla_mc_nll_backward.argtypes = [i32, i64] + [_VP] * 4
    for fn in ("kla_mc_sample", "kla_mc_sample_backward", "kla_mc_nll", "kla_mc_nll_backward"):
        getattr(lib, fn).restype = ctypes.c_int
    lib.kla_status_string.argtypes = [ctypes.c_int]
    lib.kla_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def kla_status_string(status: int) -> str:
    return _load().kla_status_string(int(status)).decode()


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _desc(q: torch.Tensor, v: torch.Tensor) -> _Desc:
    B, T, H, dk = q.shape
    return _Desc(B, T, H, dk, v.shape[-1], _DTYPES[q.dtype])


def _check_inputs(q, k, v, a, p, r):
    if not q.is_cuda:
        raise ValueError("KLA tensors must live on a GPU; the layer has no CPU path")
    if q.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {q.dtype}; use float32 or bfloat16")
    if q.dim() != 4:
        raise ValueError("q must be [B, T, H, dk]")
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (B, T, H, dk)), ("a", a, (B, T, H, dk)), ("p", p, (B, T, H, dk)),
                           ("v", v, (B, T, H, dv)), ("r", r, (B, T, H))):
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")
        if t.dtype != q.dtype or t.device != q.device:
            raise ValueError(f"{name} must share q's dtype and device")
    for name, t in (("q", q), ("k", k), ("v", v), ("a", a), ("p", p), ("r", r)):
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")


def _f32(t, shape, dev, name):
    if t is None:
        return None
    if t.dtype != torch.float32 or tuple(t.shape) != shape or t.device != dev or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {shape} on {dev}")
    return t


def kla_forward_workspace(desc: _Desc) -> int:
    return int(_load().kla_forward_workspace(ctypes.byref(desc)))


def kla_saved_bytes(desc: _Desc) -> int:
    return int(_load().kla_saved_bytes(ctypes.byref(desc)))


def kla_backward_workspace(desc: _Desc, with_saved: bool) -> int:
    return int(_load().kla_backward_workspace(ctypes.byref(desc), int(bool(with_saved))))


def kla_forward(q, k, v, a, p, r, lam0=None, eta0=None, *, want_var: bool = False,
                want_state: bool = True, save: bool = False, y=None) -> dict:
    """Filter a whole sequence.  q, k, a, p: [B, T, H, dk]; v: [B, T, H, dv];
    r: [B, T, H] (all one dtype, fp32 or bf16).  lam0 [B, H, dk], eta0
    [B, H, dk, dv] fp32 or None (prior 1 and 0).  Returns y and, as asked,
    yvar, the final belief (lamT, etaT) and the saved context for backward."""
    lib = _load()
    _check_inputs(q, k, v, a, p, r)
    dev = q.device
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    lam0 = _f32(lam0, (B, H, dk), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    desc = _desc(q, v)
    if y is None:
        y = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    yvar = torch.empty((B, T, H), dtype=torch.float32, device=dev) if want_var else None
    lamT = torch.empty((B, H, dk), dtype=torch.float32, device=dev) if want_state else None
    etaT = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_state else None
    nsaved = kla_saved_bytes(desc) if save else 0
    saved = torch.empty(max(nsaved, 1), dtype=torch.uint8, device=dev) if save else None
    nws = kla_forward_workspace(desc)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_forward(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(r), _p(lam0), _p(eta0),
                         _p(y), _p(yvar), _p(lamT), _p(etaT), _p(saved if nsaved else None), _p(ws), nws,
                         _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_forward")
    return {"y": y, "yvar": yvar, "lamT": lamT, "etaT": etaT, "saved": saved if nsaved else None}


def kla_backward(q, k, v, a, p, r, lam0, eta0, dy, dlamT=None, detaT=None, *, saved=None,
                 want_init_grads: bool = True, dyvar=None) -> dict:
    """Gradients of kla_forward's (y, yvar, lamT, etaT) for the upstream gradients
    (dy, dyvar [B, T, H] fp32 or None, dlamT, detaT); returns dq, dk, dv, da, dp,
    dr in the input dtype and, when asked, dlam0 [B, H, dk] and deta0
    [B, H, dk, dv] in fp32."""
    lib = _load()
    _check_inputs(q, k, v, a, p, r)
    dev = q.device
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    lam0 = _f32(lam0, (B, H, dk), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    dlamT = _f32(dlamT, (B, H, dk), dev, "dlamT")
    detaT = _f32(detaT, (B, H, dk, dv), dev, "detaT")
    dyvar = _f32(dyvar, (B, T, H), dev, "dyvar")
    if tuple(dy.shape) != (B, T, H, dv) or dy.dtype != q.dtype or not dy.is_contiguous():
        raise ValueError("dy must be a contiguous [B, T, H, dv] tensor in the input dtype")
    desc = _desc(q, v)
    out = {n: torch.empty_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("da", a), ("dp", p), ("dr", r))}
    dlam0 = torch.empty((B, H, dk), dtype=torch.float32, device=dev) if want_init_grads else None
    deta0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    nws = kla_backward_workspace(desc, saved is not None)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_backward(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(r), _p(lam0), _p(eta0),
                          _p(saved), _p(dy), _p(dyvar), _p(dlamT), _p(detaT), _p(out["dq"]), _p(out["dk"]), _p(out["dv"]),
                          _p(out["da"]), _p(out["dp"]), _p(out["dr"]), _p(dlam0), _p(deta0), _p(ws), nws,
                          _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_backward")
    out["dlam0"] = dlam0
    out["deta0"] = deta0
    return out


def kla_backward_noalloc(q, k, v, a, p, r, lam0, eta0, dy, dlamT=None, detaT=None, *, saved,
                         want_init_grads: bool = True, dyvar=None) -> dict:
    """kla_backward through the library's per-GPU static workspace (the entry point for
    callers that cannot allocate; only the outputs are allocated here, by torch).  A saved
    context from kla_forward(save=True) is required."""
    lib = _load()
    _check_inputs(q, k, v, a, p, r)
    dev = q.device
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    lam0 = _f32(lam0, (B, H, dk), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    dlamT = _f32(dlamT, (B, H, dk), dev, "dlamT")
    detaT = _f32(detaT, (B, H, dk, dv), dev, "detaT")
    dyvar = _f32(dyvar, (B, T, H), dev, "dyvar")
    if tuple(dy.shape) != (B, T, H, dv) or dy.dtype != q.dtype or not dy.is_contiguous():
        raise ValueError("dy must be a contiguous [B, T, H, dv] tensor in the input dtype")
    desc = _desc(q, v)
    out = {n: torch.empty_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("da", a), ("dp", p), ("dr", r))}
    dlam0 = torch.empty((B, H, dk), dtype=torch.float32, device=dev) if want_init_grads else None
    deta0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    st = lib.kla_backward_noalloc(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(r), _p(lam0), _p(eta0),
                                  _p(saved), _p(dy), _p(dyvar), _p(dlamT), _p(detaT), _p(out["dq"]), _p(out["dk"]),
                                  _p(out["dv"]), _p(out["da"]), _p(out["dp"]), _p(out["dr"]), _p(dlam0), _p(deta0),
                                  _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_backward_noalloc")
    out["dlam0"] = dlam0
    out["deta0"] = deta0
    return out


def kla_decode_step(q, k, v, a, p, r, lam, eta, *, want_var: bool = False, y=None) -> dict:
    """One token for S sequences: q, k, a, p [S, H, dk]; v [S, H, dv]; r [S, H];
    lam [S, H, dk] and eta [S, H, dk, dv] fp32 are updated in place."""
    lib = _load()
    if not q.is_cuda or q.dtype not in _DTYPES:
        raise ValueError("decode inputs must be fp32/bf16 GPU tensors")
    S, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (S, H, dk)), ("a", a, (S, H, dk)), ("p", p, (S, H, dk)),
                           ("v", v, (S, H, dv)), ("r", r, (S, H))):
        if tuple(t.shape) != shape or t.dtype != q.dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor in q's dtype")
    _f32(lam, (S, H, dk), q.device, "lam")
    _f32(eta, (S, H, dk, dv), q.device, "eta")
    if y is None:
        y = torch.empty((S, H, dv), dtype=q.dtype, device=q.device)
    yvar = torch.empty((S, H), dtype=torch.float32, device=q.device) if want_var else None
    st = lib.kla_decode_step(S, H, dk, dv, _DTYPES[q.dtype], _p(q), _p(k), _p(v), _p(a), _p(p), _p(r),
                             _p(lam), _p(eta), _p(y), _p(yvar), _stream(q.device))
    if st != 0:
        raise KLAError(st, "kla_decode_step")
    return {"y": y, "yvar": yvar, "lam": lam, "eta": eta}


def _split_grads(q, v, want_var, grads):
    """Upstream gradients of (y[, yvar], lamT, etaT) as contiguous tensors or None."""
    if want_var:
        dy, dyvar, dlamT, detaT = grads
    else:
        (dy, dlamT, detaT), dyvar = grads, None
    dy = torch.zeros_like(q[..., :1].expand(*q.shape[:3], v.shape[-1])).contiguous() if dy is None \
        else dy.contiguous()
    c = lambda t: None if t is None else t.contiguous()
    return dy, c(dyvar), c(dlamT), c(detaT)


class KLAFilter(torch.autograd.Function):
    """Autograd wrapper: y[, yvar], lamT, etaT = filter(q, k, v, a, p, r, lam0, eta0)."""

    @staticmethod
    def forward(ctx, want_var, q, k, v, a, p, r, lam0, eta0):
        out = kla_forward(q, k, v, a, p, r, lam0, eta0, want_var=want_var, want_state=True, save=True)
        ctx.save_for_backward(q, k, v, a, p, r, lam0, eta0)
        ctx.saved_ctx = out["saved"]
        ctx.want_var = want_var
        if want_var:
            return out["y"], out["yvar"], out["lamT"], out["etaT"]
        return out["y"], out["lamT"], out["etaT"]

    @staticmethod
    def backward(ctx, *grads):
        q, k, v, a, p, r, lam0, eta0 = ctx.saved_tensors
        dy, dyvar, dlamT, detaT = _split_grads(q, v, ctx.want_var, grads)
        g = kla_backward(q, k, v, a, p, r, lam0, eta0, dy, dlamT, detaT, saved=ctx.saved_ctx, dyvar=dyvar)
        return (None, g["dq"], g["dk"], g["dv"], g["da"], g["dp"], g["dr"],
                g["dlam0"] if lam0 is not None else None, g["deta0"] if eta0 is not None else None)


def kla_filter(q, k, v, a, p, r, lam0=None, eta0=None, *, want_var: bool = False):
    """Differentiable filter: returns (y, lamT, etaT), or (y, yvar, lamT, etaT)
    with want_var (the readout variance then carries a gradient too)."""
    return KLAFilter.apply(bool(want_var), q, k, v, a, p, r, lam0, eta0)


# ---- OU gates: time-invariant a, p, delta [H, dk] fp32 in place of per-token abar, pbar

def _check_ou(a, p, delta, H, dk, dev):
    for name, t in (("a", a), ("p", p), ("delta", delta)):
        _f32(t, (H, dk), dev, name)


def _check_inputs_ou(q, k, v, r):
    if not q.is_cuda:
        raise ValueError("KLA tensors must live on a GPU; the layer has no CPU path")
    if q.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {q.dtype}; use float32 or bfloat16")
    if q.dim() != 4:
        raise ValueError("q must be [B, T, H, dk]")
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (B, T, H, dk)), ("v", v, (B, T, H, dv)), ("r", r, (B, T, H))):
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {shape}")
        if t.dtype != q.dtype or t.device != q.device:
            raise ValueError(f"{name} must share q's dtype and device")
    for name, t in (("q", q), ("k", k), ("v", v), ("r", r)):
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")


def kla_backward_ou_workspace(desc: _Desc, with_saved: bool) -> int:
    return int(_load().kla_backward_ou_workspace(ctypes.byref(desc), int(bool(with_saved))))


def kla_forward_ou(q, k, v, a, p, delta, r, lam0=None, eta0=None, *, want_var: bool = False,
                   want_state: bool = True, save: bool = False, y=None) -> dict:
    """kla_forward with the gates of the OU parameters a, p, delta [H, dk] fp32."""
    lib = _load()
    _check_inputs_ou(q, k, v, r)
    dev = q.device
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    _check_ou(a, p, delta, H, dk, dev)
    lam0 = _f32(lam0, (B, H, dk), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    desc = _desc(q, v)
    if y is None:
        y = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    yvar = torch.empty((B, T, H), dtype=torch.float32, device=dev) if want_var else None
    lamT = torch.empty((B, H, dk), dtype=torch.float32, device=dev) if want_state else None
    etaT = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_state else None
    nsaved = kla_saved_bytes(desc) if save else 0
    saved = torch.empty(max(nsaved, 1), dtype=torch.uint8, device=dev) if save else None
    nws = kla_forward_workspace(desc)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_forward_ou(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(delta), _p(r), _p(lam0),
                            _p(eta0), _p(y), _p(yvar), _p(lamT), _p(etaT), _p(saved if nsaved else None), _p(ws),
                            nws, _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_forward_ou")
    return {"y": y, "yvar": yvar, "lamT": lamT, "etaT": etaT, "saved": saved if nsaved else None}


def kla_backward_ou(q, k, v, a, p, delta, r, lam0, eta0, dy, dlamT=None, detaT=None, *, saved=None,
                    want_init_grads: bool = True, dyvar=None) -> dict:
    """Gradients of kla_forward_ou (dyvar as in kla_backward): dq, dk, dv, dr in
    the input dtype; da, dp, ddelta [H, dk] fp32; dlam0, deta0 in fp32 when asked."""
    lib = _load()
    _check_inputs_ou(q, k, v, r)
    dev = q.device
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    _check_ou(a, p, delta, H, dk, dev)
    lam0 = _f32(lam0, (B, H, dk), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    dlamT = _f32(dlamT, (B, H, dk), dev, "dlamT")
    detaT = _f32(detaT, (B, H, dk, dv), dev, "detaT")
    dyvar = _f32(dyvar, (B, T, H), dev, "dyvar")
    if tuple(dy.shape) != (B, T, H, dv) or dy.dtype != q.dtype or not dy.is_contiguous():
        raise ValueError("dy must be a contiguous [B, T, H, dv] tensor in the input dtype")
    desc = _desc(q, v)
    out = {n: torch.empty_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("dr", r))}
    for n in ("da", "dp", "ddelta"):
        out[n] = torch.empty((H, dk), dtype=torch.float32, device=dev)
    dlam0 = torch.empty((B, H, dk), dtype=torch.float32, device=dev) if want_init_grads else None
    deta0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    nws = kla_backward_ou_workspace(desc, saved is not None)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_backward_ou(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(delta), _p(r), _p(lam0),
                             _p(eta0), _p(saved), _p(dy), _p(dyvar), _p(dlamT), _p(detaT), _p(out["dq"]),
                             _p(out["dk"]),
                             _p(out["dv"]), _p(out["da"]), _p(out["dp"]), _p(out["ddelta"]), _p(out["dr"]),
                             _p(dlam0), _p(deta0), _p(ws), nws, _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_backward_ou")
    out["dlam0"] = dlam0
    out["deta0"] = deta0
    return out


def kla_decode_step_ou(q, k, v, a, p, delta, r, lam, eta, *, want_var: bool = False, y=None) -> dict:
    """kla_decode_step with the gates of the OU parameters a, p, delta [H, dk] fp32."""
    lib = _load()
    if not q.is_cuda or q.dtype not in _DTYPES:
        raise ValueError("decode inputs must be fp32/bf16 GPU tensors")
    S, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (S, H, dk)), ("v", v, (S, H, dv)), ("r", r, (S, H))):
        if tuple(t.shape) != shape or t.dtype != q.dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor in q's dtype")
    _check_ou(a, p, delta, H, dk, q.device)
    _f32(lam, (S, H, dk), q.device, "lam")
    _f32(eta, (S, H, dk, dv), q.device, "eta")
    if y is None:
        y = torch.empty((S, H, dv), dtype=q.dtype, device=q.device)
    yvar = torch.empty((S, H), dtype=torch.float32, device=q.device) if want_var else None
    st = lib.kla_decode_step_ou(S, H, dk, dv, _DTYPES[q.dtype], _p(q), _p(k), _p(v), _p(a), _p(p), _p(delta),
                                _p(r), _p(lam), _p(eta), _p(y), _p(yvar), _stream(q.device))
    if st != 0:
        raise KLAError(st, "kla_decode_step_ou")
    return {"y": y, "yvar": yvar, "lam": lam, "eta": eta}


class KLAFilterOU(torch.autograd.Function):
    """Autograd wrapper: y[, yvar], lamT, etaT = filter(q, k, v, a, p, delta, r, lam0, eta0) with OU gates."""

    @staticmethod
    def forward(ctx, want_var, q, k, v, a, p, delta, r, lam0, eta0):
        out = kla_forward_ou(q, k, v, a, p, delta, r, lam0, eta0, want_var=want_var, want_state=True, save=True)
        ctx.save_for_backward(q, k, v, a, p, delta, r, lam0, eta0)
        ctx.saved_ctx = out["saved"]
        ctx.want_var = want_var
        if want_var:
            return out["y"], out["yvar"], out["lamT"], out["etaT"]
        return out["y"], out["lamT"], out["etaT"]

    @staticmethod
    def backward(ctx, *grads):
        q, k, v, a, p, delta, r, lam0, eta0 = ctx.saved_tensors
        dy, dyvar, dlamT, detaT = _split_grads(q, v, ctx.want_var, grads)
        g = kla_backward_ou(q, k, v, a, p, delta, r, lam0, eta0, dy, dlamT, detaT, saved=ctx.saved_ctx,
                            dyvar=dyvar)
        return (None, g["dq"], g["dk"], g["dv"], g["da"], g["dp"], g["ddelta"], g["dr"],
                g["dlam0"] if lam0 is not None else None, g["deta0"] if eta0 is not None else None)


def kla_filter_ou(q, k, v, a, p, delta, r, lam0=None, eta0=None, *, want_var: bool = False):
    """Differentiable filter with OU gates: returns (y, lamT, etaT), or
    (y, yvar, lamT, etaT) with want_var."""
    return KLAFilterOU.apply(bool(want_var), q, k, v, a, p, delta, r, lam0, eta0)


# ---- per-channel precision: r [B, T, H, dv], beliefs [B, H, dk, dv]

def _check_pc(q, k, v, a, p, r):
    if not q.is_cuda:
        raise ValueError("KLA tensors must live on a GPU; the layer has no CPU path")
    if q.dtype not in _DTYPES or q.dim() != 4:
        raise ValueError("q must be a [B, T, H, dk] float32 or bfloat16 tensor")
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (B, T, H, dk)), ("a", a, (B, T, H, dk)), ("p", p, (B, T, H, dk)),
                           ("v", v, (B, T, H, dv)), ("r", r, (B, T, H, dv))):
        if tuple(t.shape) != shape or t.dtype != q.dtype or t.device != q.device or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor in q's dtype")


def kla_forward_pc(q, k, v, a, p, r, lam0=None, eta0=None, *, want_var: bool = False,
                   want_state: bool = True, save: bool = False, y=None) -> dict:
    """Filter with one observation precision per value channel: q, k, a, p
    [B, T, H, dk]; v, r [B, T, H, dv] (one dtype); lam0, eta0 [B, H, dk, dv] fp32
    or None.  Returns y and, as asked, yvar [B, T, H, dv], lamT, etaT
    [B, H, dk, dv] and the saved context (belief checkpoints) for kla_backward_pc."""
    lib = _load()
    _check_pc(q, k, v, a, p, r)
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    dev = q.device
    lam0 = _f32(lam0, (B, H, dk, dv), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    desc = _desc(q, v)
    if y is None:
        y = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    yvar = torch.empty((B, T, H, dv), dtype=torch.float32, device=dev) if want_var else None
    lamT = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_state else None
    etaT = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_state else None
    nsaved = int(lib.kla_saved_pc_bytes(ctypes.byref(desc))) if save else 0
    saved = torch.empty(max(nsaved, 1), dtype=torch.uint8, device=dev) if save else None
    nws = kla_forward_workspace(desc)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_forward_pc(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(r), _p(lam0), _p(eta0),
                            _p(y), _p(yvar), _p(lamT), _p(etaT), _p(saved if nsaved else None), _p(ws), nws,
                            _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_forward_pc")
    return {"y": y, "yvar": yvar, "lamT": lamT, "etaT": etaT, "saved": saved if nsaved else None}


def kla_backward_pc(q, k, v, a, p, r, lam0, eta0, dy, dlamT=None, detaT=None, *, saved=None,
                    want_init_grads: bool = True, dyvar=None) -> dict:
    """Gradients of kla_forward_pc's (y, yvar, lamT, etaT): dq, dk, da, dp
    [B, T, H, dk] and dv, dr [B, T, H, dv] in the input dtype; dlam0, deta0
    [B, H, dk, dv] fp32 when asked.  dyvar [B, T, H, dv], dlamT, detaT
    [B, H, dk, dv] fp32 or None."""
    lib = _load()
    _check_pc(q, k, v, a, p, r)
    dev = q.device
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    lam0 = _f32(lam0, (B, H, dk, dv), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    dlamT = _f32(dlamT, (B, H, dk, dv), dev, "dlamT")
    detaT = _f32(detaT, (B, H, dk, dv), dev, "detaT")
    dyvar = _f32(dyvar, (B, T, H, dv), dev, "dyvar")
    if tuple(dy.shape) != (B, T, H, dv) or dy.dtype != q.dtype or not dy.is_contiguous():
        raise ValueError("dy must be a contiguous [B, T, H, dv] tensor in the input dtype")
    desc = _desc(q, v)
    out = {n: torch.empty_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("da", a), ("dp", p), ("dr", r))}
    dlam0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    deta0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    nws = int(lib.kla_backward_pc_workspace(ctypes.byref(desc), int(saved is not None)))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_backward_pc(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(r), _p(lam0), _p(eta0),
                             _p(saved), _p(dy), _p(dyvar), _p(dlamT), _p(detaT), _p(out["dq"]), _p(out["dk"]),
                             _p(out["dv"]), _p(out["da"]), _p(out["dp"]), _p(out["dr"]), _p(dlam0), _p(deta0),
                             _p(ws), nws, _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_backward_pc")
    out["dlam0"] = dlam0
    out["deta0"] = deta0
    return out


def kla_decode_step_pc(q, k, v, a, p, r, lam, eta, *, want_var: bool = False, y=None) -> dict:
    """One token with per-channel precision: q, k, a, p [S, H, dk]; v, r [S, H, dv];
    lam, eta [S, H, dk, dv] fp32 updated in place."""
    lib = _load()
    if not q.is_cuda or q.dtype not in _DTYPES:
        raise ValueError("decode inputs must be fp32/bf16 GPU tensors")
    S, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (S, H, dk)), ("a", a, (S, H, dk)), ("p", p, (S, H, dk)),
                           ("v", v, (S, H, dv)), ("r", r, (S, H, dv))):
        if tuple(t.shape) != shape or t.dtype != q.dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor in q's dtype")
    _f32(lam, (S, H, dk, dv), q.device, "lam")
    _f32(eta, (S, H, dk, dv), q.device, "eta")
    if y is None:
        y = torch.empty((S, H, dv), dtype=q.dtype, device=q.device)
    yvar = torch.empty((S, H, dv), dtype=torch.float32, device=q.device) if want_var else None
    st = lib.kla_decode_step_pc(S, H, dk, dv, _DTYPES[q.dtype], _p(q), _p(k), _p(v), _p(a), _p(p), _p(r),
                                _p(lam), _p(eta), _p(y), _p(yvar), _stream(q.device))
    if st != 0:
        raise KLAError(st, "kla_decode_step_pc")
    return {"y": y, "yvar": yvar, "lam": lam, "eta": eta}


# ---- block scaffolding: causal conv1d (k = 4) + SiLU, RMS QK-norm, SiLU gate

def _dense(t, name, dtype=None):
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}")
    return t


def kla_conv_silu_forward(x, w, bias=None):
    """u = silu(causal depthwise conv of x [B, T, C] with w [C, 4] (tap 3 = current token) + bias [C])."""
    lib = _load()
    _dense(x, "x")
    B, T, C = x.shape
    _f32(w, (C, 4), x.device, "w")
    _f32(bias, (C,), x.device, "bias")
    u = torch.empty_like(x)
    st = lib.kla_conv_silu_forward(B, T, C, _DTYPES[x.dtype], _p(x), _p(w), _p(bias), _p(u), _stream(x.device))
    if st != 0:
        raise KLAError(st, "kla_conv_silu_forward")
    return u


def kla_conv_silu_backward(x, w, bias, du):
    """(dx, dw, dbias) of kla_conv_silu_forward; dbias is None without a bias."""
    lib = _load()
    _dense(x, "x")
    B, T, C = x.shape
    _dense(du, "du", x.dtype)
    _f32(w, (C, 4), x.device, "w")
    _f32(bias, (C,), x.device, "bias")
    dx = torch.empty_like(x)
    dw = torch.empty((C, 4), dtype=torch.float32, device=x.device)
    db = torch.empty((C,), dtype=torch.float32, device=x.device) if bias is not None else None
    nws = int(lib.kla_conv_silu_workspace(B, T, C))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=x.device)
    st = lib.kla_conv_silu_backward(B, T, C, _DTYPES[x.dtype], _p(x), _p(w), _p(bias), _p(du), _p(dx), _p(dw),
                                    _p(db), _p(ws), nws, _stream(x.device))
    if st != 0:
        raise KLAError(st, "kla_conv_silu_backward")
    return dx, dw, db


def kla_qk_norm_forward(x, w, eps: float = 1e-6):
    """RMS normalisation of the rows (last dimension n) of x with weight w [n]; returns (out, rstd)."""
    lib = _load()
    _dense(x, "x")
    n = x.shape[-1]
    rows = x.numel() // max(n, 1)
    _f32(w, (n,), x.device, "w")
    out = torch.empty_like(x)
    rstd = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device)
    st = lib.kla_qk_norm_forward(rows, n, _DTYPES[x.dtype], _p(x), _p(w), float(eps), _p(out), _p(rstd),
                                 _stream(x.device))
    if st != 0:
        raise KLAError(st, "kla_qk_norm_forward")
    return out, rstd


def kla_qk_norm_backward(x, w, rstd, dout):
    """(dx, dw) of kla_qk_norm_forward."""
    lib = _load()
    _dense(x, "x")
    n = x.shape[-1]
    rows = x.numel() // max(n, 1)
    _f32(w, (n,), x.device, "w")
    _f32(rstd, tuple(x.shape[:-1]), x.device, "rstd")
    _dense(dout, "dout", x.dtype)
    dx = torch.empty_like(x)
    dw = torch.empty((n,), dtype=torch.float32, device=x.device)
    nws = int(lib.kla_qk_norm_workspace(n))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=x.device)
    st = lib.kla_qk_norm_backward(rows, n, _DTYPES[x.dtype], _p(x), _p(w), _p(rstd), _p(dout), _p(dx), _p(dw),
                                  _p(ws), nws, _stream(x.device))
    if st != 0:
        raise KLAError(st, "kla_qk_norm_backward")
    return dx, dw


def kla_gate_forward(y, z):
    """y * silu(z), elementwise."""
    lib = _load()
    _dense(y, "y")
    _dense(z, "z", y.dtype)
    out = torch.empty_like(y)
    st = lib.kla_gate_forward(y.numel(), _DTYPES[y.dtype], _p(y), _p(z), _p(out), _stream(y.device))
    if st != 0:
        raise KLAError(st, "kla_gate_forward")
    return out


def kla_gate_backward(y, z, dout):
    """(dy, dz) of kla_gate_forward."""
    lib = _load()
    _dense(y, "y")
    _dense(z, "z", y.dtype)
    _dense(dout, "dout", y.dtype)
    dy = torch.empty_like(y)
    dz = torch.empty_like(y)
    st = lib.kla_gate_backward(y.numel(), _DTYPES[y.dtype], _p(y), _p(z), _p(dout), _p(dy), _p(dz),
                               _stream(y.device))
    if st != 0:
        raise KLAError(st, "kla_gate_backward")
    return dy, dz


# ------------------------------------------------------------------ Monte Carlo readout (KLA+)
def _check_mc(ymu, yvar):
    if not ymu.is_cuda or ymu.dtype not in _DTYPES or ymu.dim() != 4 or not ymu.is_contiguous():
        raise ValueError("ymu must be a contiguous [B, T, H, dv] fp32/bf16 GPU tensor")
    B, T, H, dv = ymu.shape
    _f32(yvar, (B, T, H), ymu.device, "yvar")
    return B, T, H, dv


def kla_mc_sample(ymu, yvar, S: int, seed: int):
    """S draws ymu + sqrt(yvar) eps of the posterior readout: [S, B, T, H, dv] in ymu's dtype."""
    lib = _load()
    B, T, H, dv = _check_mc(ymu, yvar)
    ys = torch.empty((S, B, T, H, dv), dtype=ymu.dtype, device=ymu.device)
    st = lib.kla_mc_sample(S, B, T, H, dv, _DTYPES[ymu.dtype], int(seed) & (2**64 - 1), _p(ymu), _p(yvar), _p(ys),
                           _stream(ymu.device))
    if st != 0:
        raise KLAError(st, "kla_mc_sample")
    return ys


def kla_mc_sample_backward(yvar, dys, seed: int):
    """(dymu, dyvar) of kla_mc_sample for the gradient dys [S, B, T, H, dv] of the draws."""
    lib = _load()
    if not dys.is_cuda or dys.dtype not in _DTYPES or dys.dim() != 5 or not dys.is_contiguous():
        raise ValueError("dys must be a contiguous [S, B, T, H, dv] fp32/bf16 GPU tensor")
    S, B, T, H, dv = dys.shape
    _f32(yvar, (B, T, H), dys.device, "yvar")
    dymu = torch.empty((B, T, H, dv), dtype=dys.dtype, device=dys.device)
    dyvar = torch.empty((B, T, H), dtype=torch.float32, device=dys.device)
    st = lib.kla_mc_sample_backward(S, B, T, H, dv, _DTYPES[dys.dtype], int(seed) & (2**64 - 1), _p(yvar), _p(dys),
                                    _p(dymu), _p(dyvar), _stream(dys.device))
    if st != 0:
        raise KLAError(st, "kla_mc_sample_backward")
    return dymu, dyvar


def kla_mc_nll(logp):
    """-logsumexp_s(logp[s]) + log S per token, logp [S, n] fp32 (the decoder's log-probabilities of
    the target tokens under each draw)."""
    lib = _load()
    _dense(logp, "logp", torch.float32)
    S = logp.shape[0]
    n = logp.numel() // S
    nll = torch.empty(logp.shape[1:], dtype=torch.float32, device=logp.device)
    st = lib.kla_mc_nll(S, n, _p(logp), _p(nll), _stream(logp.device))
    if st != 0:
        raise KLAError(st, "kla_mc_nll")
    return nll


def kla_mc_nll_backward(logp, dnll):
    """dlogp = -dnll softmax over the draws, [S, n] fp32."""
    lib = _load()
    _dense(logp, "logp", torch.float32)
    _dense(dnll, "dnll", torch.float32)
    S = logp.shape[0]
    n = logp.numel() // S
    if dnll.numel() != n:
        raise ValueError("dnll must hold one value per token")
    dlogp = torch.empty_like(logp)
    st = lib.kla_mc_nll_backward(S, n, _p(logp), _p(dnll), _p(dlogp), _stream(logp.device))
    if st != 0:
        raise KLAError(st, "kla_mc_nll_backward")
    return dlogp


class KLAMCSample(torch.autograd.Function):
    """Autograd wrapper: ys = draws(ymu, yvar); the seed selects the draws."""

    @staticmethod
    def forward(ctx, ymu, yvar, S, seed):
        ymu_c, yvar_c = ymu.contiguous(), yvar.contiguous()
        ctx.save_for_backward(yvar_c)
        ctx.seed = seed
        return kla_mc_sample(ymu_c, yvar_c, S, seed)

    @staticmethod
    def backward(ctx, dys):
        (yvar,) = ctx.saved_tensors
        dymu, dyvar = kla_mc_sample_backward(yvar, dys.contiguous(), ctx.seed)
        return dymu, dyvar, None, None


class KLAMCNLL(torch.autograd.Function):
    """Autograd wrapper: nll = -logsumexp_s(logp) + log S."""

    @staticmethod
    def forward(ctx, logp):
        logp_c = logp.contiguous()
        ctx.save_for_backward(logp_c)
        return kla_mc_nll(logp_c)

    @staticmethod
    def backward(ctx, dnll):
        (logp,) = ctx.saved_tensors
        return kla_mc_nll_backward(logp, dnll.contiguous())


def kla_mc_nll_loss(ymu, yvar, decoder_logp, S: int = 10, seed: int = 0):
    """The KLA+ objective per token: draws of the readout, the decoder's log-probability of
    the targets under each draw (decoder_logp: a function of [S, B, T, H, dv] draws returning
    [S, ...] fp32 log-probabilities, part of the model), and -logsumexp over the draws + log S."""
    ys = KLAMCSample.apply(ymu, yvar, S, seed)
    return KLAMCNLL.apply(decoder_logp(ys))


# ------------------------------------------------------------------ gates per (key slot, value channel)
def _check_pc_ou(q, k, v, r, a, p, delta):
    if not q.is_cuda or q.dtype not in _DTYPES:
        raise ValueError("inputs must be fp32/bf16 GPU tensors")
    B, T, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (B, T, H, dk)), ("v", v, (B, T, H, dv)), ("r", r, (B, T, H, dv))):
        if tuple(t.shape) != shape or t.dtype != q.dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor in q's dtype")
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    for name, t in (("a", a), ("p", p), ("delta", delta)):
        _f32(t, (H, dk, dv), q.device, name)
    return B, T, H, dk, dv


def kla_forward_pc_ou(q, k, v, a, p, delta, r, lam0=None, eta0=None, *, want_var: bool = False,
                      want_state: bool = True, save: bool = False) -> dict:
    """Filter with gates per (key slot, value channel) from OU parameters a, p, delta
    [H, dk, dv] fp32 and one observation precision per value channel r [B, T, H, dv]
    (Algorithm 1's shapes).  Returns as kla_forward_pc."""
    lib = _load()
    B, T, H, dk, dv = _check_pc_ou(q, k, v, r, a, p, delta)
    dev = q.device
    lam0 = _f32(lam0, (B, H, dk, dv), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    desc = _desc(q, v)
    y = torch.empty((B, T, H, dv), dtype=q.dtype, device=dev)
    yvar = torch.empty((B, T, H, dv), dtype=torch.float32, device=dev) if want_var else None
    lamT = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_state else None
    etaT = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_state else None
    nsaved = int(lib.kla_saved_pc_bytes(ctypes.byref(desc))) if save else 0
    saved = torch.empty(max(nsaved, 1), dtype=torch.uint8, device=dev) if save else None
    nws = kla_forward_workspace(desc)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_forward_pc_ou(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(delta), _p(r), _p(lam0),
                               _p(eta0), _p(y), _p(yvar), _p(lamT), _p(etaT), _p(saved if nsaved else None), _p(ws),
                               nws, _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_forward_pc_ou")
    return {"y": y, "yvar": yvar, "lamT": lamT, "etaT": etaT, "saved": saved if nsaved else None}


def kla_backward_pc_ou(q, k, v, a, p, delta, r, lam0, eta0, dy, dlamT=None, detaT=None, *, saved=None,
                       want_init_grads: bool = True, dyvar=None) -> dict:
    """Gradients of kla_forward_pc_ou: dq, dk [B, T, H, dk] and dv, dr [B, T, H, dv] in the
    input dtype; da, dp, ddelta [H, dk, dv] fp32; dlam0, deta0 [B, H, dk, dv] when asked."""
    lib = _load()
    B, T, H, dk, dv = _check_pc_ou(q, k, v, r, a, p, delta)
    dev = q.device
    lam0 = _f32(lam0, (B, H, dk, dv), dev, "lam0")
    eta0 = _f32(eta0, (B, H, dk, dv), dev, "eta0")
    dlamT = _f32(dlamT, (B, H, dk, dv), dev, "dlamT")
    detaT = _f32(detaT, (B, H, dk, dv), dev, "detaT")
    dyvar = _f32(dyvar, (B, T, H, dv), dev, "dyvar")
    if tuple(dy.shape) != (B, T, H, dv) or dy.dtype != q.dtype or not dy.is_contiguous():
        raise ValueError("dy must be a contiguous [B, T, H, dv] tensor in the input dtype")
    desc = _desc(q, v)
    out = {n: torch.empty_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("dr", r))}
    for n in ("da", "dp", "ddelta"):
        out[n] = torch.empty((H, dk, dv), dtype=torch.float32, device=dev)
    dlam0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    deta0 = torch.empty((B, H, dk, dv), dtype=torch.float32, device=dev) if want_init_grads else None
    nws = int(lib.kla_backward_pc_ou_workspace(ctypes.byref(desc), int(saved is not None)))
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    st = lib.kla_backward_pc_ou(ctypes.byref(desc), _p(q), _p(k), _p(v), _p(a), _p(p), _p(delta), _p(r), _p(lam0),
                                _p(eta0), _p(saved), _p(dy), _p(dyvar), _p(dlamT), _p(detaT), _p(out["dq"]),
                                _p(out["dk"]), _p(out["dv"]), _p(out["da"]), _p(out["dp"]), _p(out["ddelta"]),
                                _p(out["dr"]), _p(dlam0), _p(deta0), _p(ws), nws, _stream(dev))
    if st != 0:
        raise KLAError(st, "kla_backward_pc_ou")
    out["dlam0"] = dlam0
    out["deta0"] = deta0
    return out


def kla_decode_step_pc_ou(q, k, v, a, p, delta, r, lam, eta, *, want_var: bool = False, y=None) -> dict:
    """One token for S sequences with gates per (key slot, value channel): q, k [S, H, dk];
    v, r [S, H, dv]; a, p, delta [H, dk, dv]; lam, eta [S, H, dk, dv] fp32 updated in place."""
    lib = _load()
    S, H, dk = q.shape
    dv = v.shape[-1]
    for name, t, shape in (("k", k, (S, H, dk)), ("v", v, (S, H, dv)), ("r", r, (S, H, dv))):
        if tuple(t.shape) != shape or t.dtype != q.dtype or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous {shape} tensor in q's dtype")
    for name, t in (("a", a), ("p", p), ("delta", delta)):
        _f32(t, (H, dk, dv), q.device, name)
    _f32(lam, (S, H, dk, dv), q.device, "lam")
    _f32(eta, (S, H, dk, dv), q.device, "eta")
    if y is None:
        y = torch.empty((S, H, dv), dtype=q.dtype, device=q.device)
    yvar = torch.empty((S, H, dv), dtype=torch.float32, device=q.device) if want_var else None
    st = lib.kla_decode_step_pc_ou(S, H, dk, dv, _DTYPES[q.dtype], _p(q), _p(k), _p(v), _p(a), _p(p), _p(delta),
                                   _p(r), _p(lam), _p(eta), _p(y), _p(yvar), _stream(q.device))
    if st != 0:
        raise KLAError(st, "kla_decode_step_pc_ou")
    return {"y": y, "yvar": yvar, "lam": lam, "eta": eta}


class KLAFilterPcOU(torch.autograd.Function):
    """Autograd wrapper: y, lamT, etaT = filter(q, k, v, a, p, delta, r) with gates per
    (key slot, value channel) from OU parameters [H, dk, dv]."""

    @staticmethod
    def forward(ctx, q, k, v, a, p, delta, r):
        out = kla_forward_pc_ou(q, k, v, a, p, delta, r, save=True)
        ctx.save_for_backward(q, k, v, a, p, delta, r, out["saved"])
        return out["y"], out["lamT"], out["etaT"]

    @staticmethod
    def backward(ctx, dy, dlamT, detaT):
        q, k, v, a, p, delta, r, saved = ctx.saved_tensors
        c = lambda t: None if t is None else t.contiguous()
        dy = torch.zeros_like(q[..., :1].expand(*q.shape[:3], v.shape[-1])).contiguous() if dy is None \
            else dy.contiguous()
        g = kla_backward_pc_ou(q, k, v, a, p, delta, r, None, None, dy, c(dlamT), c(detaT), saved=saved,
                               want_init_grads=False)
        return g["dq"], g["dk"], g["dv"], g["da"], g["dp"], g["ddelta"], g["dr"]


def kla_filter_pc_ou(q, k, v, a, p, delta, r):
    return KLAFilterPcOU.apply(q, k, v, a, p, delta, r)
