"""Seeded synthetic inputs for the KLA filter layer (shared by tests, bench and oracle).

This module draws random numbers and shapes them into the input distributions of
the five workloads; it holds none of the filter's arithmetic.  Every tensor is
drawn in float64 from ``numpy.random.default_rng([seed, tensor_id, b, h])`` so that
any (batch, head) slice can be regenerated on its own, then quantised once to the
workload's dtype.  Both the GPU path and the oracle consume the *quantised*
values (the oracle widened back to float64).

Quantisation: float64 -> float32 with numpy's round-to-nearest-even, then, for
bf16, float32 -> bf16 by round-to-nearest-even on the bit pattern.

Tensor names follow the paper's notation: ``q`` query (readout operator), ``k``
key (observation operator), ``v`` value (observation), ``a`` the discretised
decay abar in (0, 1], ``p`` the discretised process-noise variance pbar >= 0, ``r``
the observation (value) precision Lambda^v > 0, one per token and head, and
``dy`` the upstream gradient of the output.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from functools import lru_cache
from typing import Iterable, Optional

import numpy as np

TENSOR_ID = {"q": 0, "k": 1, "v": 2, "a": 3, "p": 4, "r": 5, "dy": 6, "rc": 10}
KEY_DIM = ("q", "k", "a", "p")          # [B, T, H, dk]
VAL_DIM = ("v", "dy", "rc")             # [B, T, H, dv]; rc: one observation precision per value channel
NAMES = ("q", "k", "v", "a", "p", "r")


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def softplus(x):
    return np.log1p(np.exp(-np.abs(x))) + np.maximum(x, 0.0)


def to_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64/float32 -> bf16 bit patterns (uint16), round-to-nearest-even."""
    f = np.ascontiguousarray(to_f32(x))
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def quantise(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to ``dtype`` ('f32' or 'bf16') and widen back to float64."""
    if dtype == "f32":
        return to_f32(x).astype(np.float64)
    if dtype == "bf16":
        return bf16_to_f64(bf16_bits(x))
    raise ValueError(dtype)


@dataclass(frozen=True)
class Workload:
    """One of the five workload shapes (batch B, heads H, length T, key/value widths)."""
    cid: int
    name: str
    B: int
    T: int
    H: int
    dk: int
    dv: int
    dtype: str                      # 'f32' or 'bf16'
    dist: str                       # 'c0' | 'a5' | 'lm' | 'long'
    backward: bool
    extra: dict = field(default_factory=dict)

    @property
    def token_heads(self) -> int:
        return self.B * self.T * self.H


WORKLOADS = {
    0: Workload(0, "tiny_fwd_f32", 1, 256, 2, 16, 16, "f32", "c0", False),
    1: Workload(1, "a5_state_tracking_f32", 64, 512, 4, 32, 32, "f32", "a5", True,
                {"vocab": 60, "d_model": 128}),
    2: Workload(2, "lm_layer_1p3b_bf16", 8, 2048, 16, 128, 128, "bf16", "lm", True),
    3: Workload(3, "long_context_64k_bf16", 1, 65536, 16, 128, 128, "bf16", "long", False),
    # decode: S sequences, a 1024-token prewarm forward then 256 single-token steps
    4: Workload(4, "decode_512x16_f32", 512, 1024, 16, 128, 128, "f32", "lm", False,
                {"steps": 256}),
}


def _rng(seed: int, tid: int, b: int, h: int) -> np.random.Generator:
    return np.random.default_rng([seed, tid, b, h])


def _draw_iid(w: Workload, name: str, b: int, h: int, T: int, seed: int) -> np.ndarray:
    """float64 draws for one (b, h) slice, before quantisation: [T, width]."""
    width = w.dk if name in KEY_DIM else (w.dv if name in VAL_DIM else 1)
    g = _rng(seed, TENSOR_ID[name], b, h)
    z = g.standard_normal((T, width))
    if w.dist == "c0":
        if name in ("q", "k"):
            return z / np.sqrt(w.dk)
        if name in ("v", "dy"):
            return z
        if name == "a":
            return sigmoid(z + 2.0)
        if name == "p":
            return softplus(z - 2.0)
        return softplus(z)                      # r, rc
    # language-model distributions (also the long-context stress)
    if name == "k":
        return z / np.linalg.norm(z, axis=1, keepdims=True)
    if name in ("q", "v", "dy"):
        return z
    if name == "a":
        shift = 6.0 if (w.dist == "long" and h >= w.H // 2) else 3.0
        return sigmoid(z + shift)
    if name == "p":
        return softplus(z - 3.0)
    return softplus(z)                          # r, rc


@lru_cache(maxsize=4)
def _a5_tables(seed: int, V: int, dm: int, ncol: int):
    """Embedding table E [V, d_model] ~ N(0, 1) and projection W [d_model, ncol] ~ N(0, 1/d_model)."""
    E = _rng(seed, 101, 0, 0).standard_normal((V, dm))
    W = _rng(seed, 102, 0, 0).standard_normal((dm, ncol)) / np.sqrt(dm)
    return E, W


def _a5_block(w: Workload, b: int, T: int, seed: int) -> np.ndarray:
    """Token-embedding projection for one batch row: [T, 4*H*dk + H*dv + H]."""
    V, dm = w.extra["vocab"], w.extra["d_model"]
    E, W = _a5_tables(seed, V, dm, 4 * w.H * w.dk + w.H * w.dv + w.H)
    x = _rng(seed, 100, b, 0).integers(0, V, size=T)
    return E[x] @ W


def _a5_slice(w: Workload, name: str, proj: np.ndarray, h: int) -> np.ndarray:
    H, dk, dv = w.H, w.dk, w.dv
    off = {"q": 0, "k": H * dk, "v": 2 * H * dk, "a": 2 * H * dk + H * dv,
           "p": 3 * H * dk + H * dv, "r": 4 * H * dk + H * dv}[name]
    width = dv if name == "v" else (1 if name == "r" else dk)
    z = proj[:, off + h * width: off + (h + 1) * width]
    if name in ("q", "k"):
        return z / np.sqrt(dk)
    if name == "v":
        return z
    if name == "a":
        return sigmoid(2.0 + z)
    if name == "p":
        return softplus(-2.0 + z)
    return softplus(z)


def draw(w: Workload, name: str, b: int, h: int, seed: Optional[int] = None,
         T: Optional[int] = None, proj_cache: Optional[dict] = None) -> np.ndarray:
    """Quantised float64 values of one (b, h) slice: [T, width] ([T] for r)."""
    seed = w.cid if seed is None else seed
    T = w.T if T is None else T
    if w.dist == "a5" and name != "dy":
        key = (seed, b, T)
        if proj_cache is not None and key in proj_cache:
            proj = proj_cache[key]
        else:
            proj = _a5_block(w, b, T, seed)
            if proj_cache is not None:
                proj_cache.clear()
                proj_cache[key] = proj
        x = _a5_slice(w, name, proj, h)
    else:
        x = _draw_iid(w, name, b, h, T, seed)
    x = quantise(x, w.dtype)
    return x[:, 0] if name == "r" else x


def full(w: Workload, names: Iterable[str] = NAMES + ("dy",), seed: Optional[int] = None,
         T: Optional[int] = None, as_bits: bool = False, threads: Optional[int] = None) -> dict:
    """All (b, h) slices assembled into [B, T, H, width] arrays ([B, T, H] for r).

    ``as_bits=True`` returns the storage form (float32, or uint16 bf16 bit
    patterns) for upload; otherwise float64 holding the quantised values.
    Slices are drawn on a thread pool; the values do not depend on it."""
    T = w.T if T is None else T
    if threads is None:
        try:
            threads = min(16, len(os.sched_getaffinity(0)))
        except AttributeError:  # pragma: no cover
            threads = 4
    out = {}
    for name in names:
        width = w.dk if name in KEY_DIM else (w.dv if name in VAL_DIM else None)
        shape = (w.B, T, w.H) + ((width,) if width else ())
        if as_bits:
            arr = np.empty(shape, dtype=np.uint16 if w.dtype == "bf16" else np.float32)
        else:
            arr = np.empty(shape, dtype=np.float64)

        def fill(task, name=name, arr=arr):
            b, hs = task
            cache: dict = {}
            for h in hs:
                x = draw(w, name, b, h, seed=seed, T=T, proj_cache=cache)
                if as_bits:
                    x = bf16_bits(x) if w.dtype == "bf16" else to_f32(x)
                arr[b, :, h] = x

        # the token-projection workload shares one projection per batch row
        if w.dist == "a5":
            tasks = [(b, range(w.H)) for b in range(w.B)]
        else:
            tasks = [(b, (h,)) for b in range(w.B) for h in range(w.H)]
        if threads > 1 and len(tasks) > 1:
            with ThreadPoolExecutor(max_workers=threads) as ex:
                list(ex.map(fill, tasks))
        else:
            for task in tasks:
                fill(task)
        out[name] = arr
    return out


def pairs_slice(w: Workload, pairs, names: Iterable[str] = NAMES + ("dy",),
                seed: Optional[int] = None, T: Optional[int] = None) -> dict:
    """Selected (b, h) pairs as float64 arrays shaped [len(pairs), T, 1, width]
    (r: [len(pairs), T, 1]) -- independent sequences for the oracle."""
    out = {}
    cache: dict = {}
    for name in names:
        rows = [draw(w, name, b, h, seed=seed, T=T, proj_cache=cache) for (b, h) in pairs]
        arr = np.stack(rows)[:, :, None]
        out[name] = arr
    return out


def random_case(B: int, T: int, H: int, dk: int, dv: int, dtype: str = "f32",
                seed: int = 1234, dist: str = "c0") -> dict:
    """A seeded case of any shape with a named workload's distributions."""
    w = Workload(-1, "custom", B, T, H, dk, dv, dtype, dist, True)
    return full(w, seed=seed)


def decode_inputs(w: Workload, seed: Optional[int] = None, as_bits: bool = False) -> dict:
    """Per-step inputs of the decode workload: [S, steps, H, width] float64
    (the steps are drawn as a second sequence, with the seed offset by 1000)."""
    seed = w.cid if seed is None else seed
    steps = w.extra["steps"]
    w2 = Workload(w.cid, w.name, w.B, steps, w.H, w.dk, w.dv, w.dtype, w.dist, False)
    return full(w2, names=NAMES, seed=seed + 1000, as_bits=as_bits)


OU_TENSOR_ID = {"a": 7, "p": 8, "delta": 9}


def ou_params(H: int, dk: int, seed: int = 0, dv: Optional[int] = None) -> dict:
    """Time-invariant OU parameters [H, dk] (or [H, dk, dv] when dv is given: one per
    key slot and value channel) as float32 (the storage form; the oracle widens
    them): step size delta log-uniform on [1e-3, 1e-1], mean reversion a uniform on
    [1, 16], diffusion scale p = softplus(N(2, 1)).  The resulting decays
    exp(-a delta) span about (0.2, 0.999), centred near 0.92."""
    out = {}
    shape = (dk,) if dv is None else (dk, dv)
    for name, tid in OU_TENSOR_ID.items():
        rows = []
        for h in range(H):
            g = _rng(seed, tid + (0 if dv is None else 10), 0, h)
            if name == "delta":
                x = np.exp(g.uniform(np.log(1e-3), np.log(1e-1), shape))
            elif name == "a":
                x = g.uniform(1.0, 16.0, shape)
            else:
                x = softplus(g.standard_normal(shape) + 2.0)
            rows.append(x)
        out[name] = to_f32(np.stack(rows))
    return out
