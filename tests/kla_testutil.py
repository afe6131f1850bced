"""Helpers shared by the GPU parity tests: tolerance metric and tensor plumbing."""
import os

import numpy as np

# Tolerances on the floored relative error below: fp32 inputs, bf16 inputs with
# fp32 state and accumulation.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_err(x, ref, floor_frac: float = 1.0) -> float:
    """max_i |x_i - r_i| / max(|r_i|, floor_frac * rms(r)).

    The gate uses floor_frac = 1: an element at least as large as the tensor's
    rms is judged relative to itself, a smaller one (the result of cancellation
    between terms of rms size, whose rounding error scales with the rms) relative
    to the rms.  floor_frac = 0.01 gives the stricter figure also reported."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref * ref))
    floor = max(floor_frac * rms, 1e-300)
    return float(np.max(np.abs(x - ref) / np.maximum(np.abs(ref), floor)))


def to_torch(arr, dtype: str, device):
    """float64 numpy (already quantised) -> device tensor in the storage dtype."""
    import torch
    import kla_inputs as K
    if dtype == "bf16":
        bits = K.bf16_bits(arr).view(np.int16)
        return torch.from_numpy(np.ascontiguousarray(bits)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr.astype(np.float32))).to(device)


def bits_to_torch(bits, device):
    import torch
    if bits.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(bits.view(np.int16))).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(bits)).to(device)


def to_np(t) -> np.ndarray:
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def log(msg: str):
    print(msg, flush=True)
