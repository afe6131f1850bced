"""Helpers shared by the GPU parity tests: tolerance metric and tensor plumbing."""
import os

import numpy as np

# Tolerances on the floored relative error below: fp32 inputs, bf16 inputs with
# fp32 state and accumulation.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_err(x, ref, floor_frac: float = 0.01) -> float:
    """max_i |x_i - r_i| / max(|r_i|, floor_frac * rms(r)).

    The gate uses floor_frac = 0.01: an element is judged relative to itself
    unless it is smaller than 1% of the tensor's rms, where the floor stands in
    for it (a near-zero element is the result of cancellation between terms of
    rms size, whose rounding error scales with the rms).  floor_frac = 1 gives
    the rms-relative figure also reported."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref * ref))
    floor = max(floor_frac * rms, 1e-300)
    return float(np.max(np.abs(x - ref) / np.maximum(np.abs(ref), floor)))


def rel_err_sum(x, ref, mass, floor_frac: float = 0.01) -> float:
    """rel_err for a tensor each of whose elements is a sum over (b, t) of per-token
    terms (the gradient of a parameter shared by every token): the error of an
    element is judged against max(|r_i|, floor_frac * rms(r), mass_i), where mass_i is
    the sum of the absolute values of its terms.  A sum of terms each accurate to a
    relative delta is accurate to delta * mass; with heavy cancellation (|r_i| much
    smaller than mass_i) that, and not |r_i|, is the scale of its rounding."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    mass = np.asarray(mass, dtype=np.float64)
    assert x.shape == ref.shape == mass.shape, (x.shape, ref.shape, mass.shape)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref * ref))
    floor = np.maximum(max(floor_frac * rms, 1e-300), mass)
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
