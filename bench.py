"""Throughput of the KLA filter layer (forward + backward) on one MI355X.

One step = kla_forward (saving the context for backward) + kla_backward over
one batch of the language-model layer workload (B=8, H=16, T=2048,
d_k=d_v=128, bf16 inputs with fp32 state), inputs already resident in HBM.
The value is token-heads (B*T*H) per second.

Besides the JSON line's throughput it reports, for the dominant call (the
backward: kernels bwd_dv, bwd_dk and dr_combine), the achieved fraction of
the HBM roofline from the algorithmic bytes per call and that call's average
duration taken with HIP events on the stream it runs on; the measured HBM
traffic of that call when profiles/lm_layer_traffic.md was taken from the
current kernel sources (see paper_2602_10743_amd/traffic.py); and the fp64
oracle's throughput on the host cores over a bounded sample of the same
workload.

With --ou the same shape runs with OU gates instead (kla_forward_ou /
kla_backward_ou: time-invariant a, p, delta [H, dk] in place of the per-token
abar and pbar tensors); its traffic summary is profiles/lm_layer_ou_traffic.md.

With --pc it times forward + backward of the per-channel-precision variant
(kla_forward_pc / kla_backward_pc: r drawn per value channel, precision and
gates per (key slot, value channel)), elementwise scans bound by VALU issue;
their roofline is the chip's fp32 VALU issue rate (see ALU_SLOTS_*).

With --decode it times kla_decode_step on the decode workload (S = 512
sequences, H = 16, d = 128, fp32 belief of 512 MiB updated in place), HBM-bound
on the belief; --decode --pc times kla_decode_step_pc (per-channel precision:
the precision is a second dk x dv array per head).

With --long it times the forward of the long-context workload (B = 1, H = 16,
T = 65536, d = 128, bf16; heads 8..15 with slow decay), which has only 16
sequences to spread over the chip.

With --a5 it times forward + backward of the state-tracking workload (B = 64,
H = 4, T = 512, d = 32, fp32 inputs: the chunked fp64 kernels).

With --mc it times the Monte Carlo readout of KLA+ at the same shape with S = 10
draws: kla_mc_sample, kla_mc_sample_backward, kla_mc_nll and kla_mc_nll_backward.

With --block it times the block scaffolding around the layer at the same shape,
forward + backward: the causal conv1d + SiLU over the C = H dk channels, the
RMS QK-norm of q and of k (rows of dk) and the SiLU gate of the output, all
HBM-bound; the roofline object is for the dominant kernel call.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np

METRIC = "KLA layer fwd+bwd tokens/sec (B·T·H, d=128) on 1 MI355X; % of HBM/MFMA roofline"
HBM_PEAK_GBS = 8000.0
# fp32 VALU issue of the chip: 256 CUs x 4 SIMDs, one wave64 instruction (64 lanes) per 4
# cycles per SIMD at 2.4 GHz, i.e. 16 lane-operations per cycle per SIMD (packed fp32 unused)
VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9
# issue slots of one element update of the per-channel scan, with the per-token products
# abar^2, k^2, q^2 and r v shared by a row or column: den = abar^2 + pbar lam (1), k^2 r (1),
# num = lam + k^2 r den (1), den num (1), its reciprocal R (quarter rate: 4), 1/den = num R and
# lam_t = num / den (2), 1/lam_t = den^2 R (2), the gate abar / den (1), k r v (1), eta_t (1),
# eta_t / lam_t (1) and the two readout sums (2)
ALU_SLOTS_PER_ELEMENT = 18
# backward, per element and token: the recomputed update (13 slots: the forward's without the
# readouts) and the adjoint step as written in pc.hip with the same sharing (38 slots, one
# quarter-rate reciprocal of lam_t den among them)
ALU_SLOTS_BWD_PER_ELEMENT = 51


def algorithmic_bytes(w, s, ou=False):
    """Per token-head: forward reads q,k,abar,pbar (dk each), v (dv), r (1) and
    writes y (dv); backward reads those plus dy and writes the six gradients.
    With OU gates there are no per-token abar, pbar or their gradients (the
    [H, dk] parameters and their gradients are a fixed few KiB per call)."""
    nk = 2 if ou else 4
    fwd = (nk * w.dk + w.dv + 1) * s + w.dv * s
    bwd = 2 * (nk * w.dk + w.dv + 1) * s + w.dv * s
    return fwd, bwd


def cpu_baseline_pc(w):
    """fp64 oracle forward + backward of the per-channel workload on a few sampled sequences."""
    import kla_inputs as K
    import oracle
    threads = oracle.default_threads()
    pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
    np.random.default_rng(0).shuffle(pairs)
    sample = sorted(pairs[:max(1, min(2 * threads, len(pairs)))])
    sl = K.pairs_slice(w, sample, names=("q", "k", "v", "a", "p", "rc", "dy"))
    t0 = time.perf_counter()
    oracle.forward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["rc"], nthreads=threads)
    t1 = time.perf_counter()
    oracle.backward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["rc"], None, None, sl["dy"], nthreads=threads)
    t2 = time.perf_counter()
    return {"value": len(sample) * w.T / (t2 - t0), "unit": "tokens/s", "cores": min(threads, len(sample)),
            "kind": "oracle",
            "sample": f"{len(sample)} (batch, head) sequences of T={w.T} (fwd {t1 - t0:.1f}s + bwd {t2 - t1:.1f}s)"}


def bench_pc(args, w, dev):
    """Forward + backward of the per-channel-precision variant at the LM-layer shape; with
    --ou its gates per (key slot, value channel) come from OU parameters [H, dk, dv]
    (kla_forward_pc_ou / kla_backward_pc_ou, Algorithm 1's shapes)."""
    import torch
    import kla_inputs as K
    import paper_2602_10743_amd as kla
    names = ("q", "k", "v", "rc", "dy") if args.ou else ("q", "k", "v", "a", "p", "rc", "dy")
    bits = K.full(w, names=names, as_bits=True)
    x = {n: torch.from_numpy(np.ascontiguousarray(bits[n].view(np.int16))).view(torch.bfloat16).to(dev)
         for n in bits}
    del bits
    ou = None
    if args.ou:
        ou = {n: torch.from_numpy(v).to(dev) for n, v in K.ou_params(w.H, w.dk, seed=w.cid, dv=w.dv).items()}
    stream = torch.cuda.current_stream(dev)
    y = torch.empty_like(x["v"])

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        if ou is None:
            out = kla.kla_forward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], want_state=False, save=True,
                                     y=y)
        else:
            out = kla.kla_forward_pc_ou(x["q"], x["k"], x["v"], ou["a"], ou["p"], ou["delta"], x["rc"],
                                        want_state=False, save=True)
        if ev is not None:
            ev[1].record(stream)
        if ou is None:
            kla.kla_backward_pc(x["q"], x["k"], x["v"], x["a"], x["p"], x["rc"], None, None, x["dy"],
                                saved=out["saved"], want_init_grads=False)
        else:
            kla.kla_backward_pc_ou(x["q"], x["k"], x["v"], ou["a"], ou["p"], ou["delta"], x["rc"], None, None,
                                   x["dy"], saved=out["saved"], want_init_grads=False)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    bwd_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    th = w.token_heads
    elements = th * w.dk * w.dv
    achieved = elements * ALU_SLOTS_BWD_PER_ELEMENT / (bwd_ms * 1e-3)
    res = {
        "metric": METRIC, "value": th / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name + ("_pc_ou" if ou else "_pc"), "B": w.B, "T": w.T, "H": w.H, "dk": w.dk,
                   "dv": w.dv, "pass": "fwd+bwd", "precision": "per value channel (bf16 inputs, fp32 scan)",
                   "gates": "ou (a, p, delta per head, key slot and value channel)" if ou else "per token",
                   "tokens_counted": "B*T*H"},
        "roofline": {"bound": "alu", "kernel": "kla_backward_pc_ou" if ou else "kla_backward_pc",
                     "achieved": achieved / 1e12,
                     "peak": VALU_LANE_OPS / 1e12, "unit": "T lane-ops/s",
                     "frac": achieved / VALU_LANE_OPS, "traffic": None,
                     "element_updates_per_call": elements, "slots_per_element": ALU_SLOTS_BWD_PER_ELEMENT,
                     "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
                     "fwd_frac": elements * ALU_SLOTS_PER_ELEMENT / (fwd_ms * 1e-3) / VALU_LANE_OPS},
    }
    if not args.no_cpu_baseline and ou is None:
        res["cpu_baseline"] = cpu_baseline_pc(w)
    print(json.dumps(res), flush=True)


def bench_block(args, w, dev):
    """Conv + SiLU, QK-norm (q and k) and gate, forward + backward, at the LM-layer shape."""
    import torch
    import paper_2602_10743_amd as kla
    B, T, H, d = w.B, w.T, w.H, w.dk
    C = H * d
    gen = torch.Generator(device=dev).manual_seed(0)
    r = lambda *s: torch.randn(*s, generator=gen, device=dev).to(torch.bfloat16)
    x, du, q, k, y, z, g = r(B, T, C), r(B, T, C), r(B, T, H, d), r(B, T, H, d), r(B, T, C), r(B, T, C), r(B, T, C)
    cw = torch.randn(C, 4, generator=gen, device=dev) * 0.5
    cb = torch.randn(C, generator=gen, device=dev)
    nw = torch.ones(d, device=dev)
    stream = torch.cuda.current_stream(dev)
    calls = {}

    def timed(name, fn):
        if name not in calls:
            calls[name] = []
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        out = fn()
        e1.record(stream)
        calls[name].append((e0, e1))
        return out

    def step():
        timed("conv_fwd", lambda: kla.kla_conv_silu_forward(x, cw, cb))
        timed("conv_bwd", lambda: kla.kla_conv_silu_backward(x, cw, cb, du))
        for nm, t in (("q", q), ("k", k)):
            out, rstd = timed("norm_fwd", lambda: kla.kla_qk_norm_forward(t, nw, 1e-6))
            timed("norm_bwd", lambda: kla.kla_qk_norm_backward(t, nw, rstd, out))
        timed("gate_fwd", lambda: kla.kla_gate_forward(y, z))
        timed("gate_bwd", lambda: kla.kla_gate_backward(y, z, g))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    calls.clear()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = {n: float(np.mean([a.elapsed_time(b) for a, b in v])) for n, v in calls.items()}
    th = w.token_heads
    s = 2
    # algorithmic bytes per call (bf16 tensors; fp32 row statistics and weights are negligible)
    nbytes = {"conv_fwd": 2 * B * T * C * s, "conv_bwd": 3 * B * T * C * s,
              "norm_fwd": 2 * th * d * s + th * 4, "norm_bwd": 3 * th * d * s + th * 4,
              "gate_fwd": 3 * B * T * C * s, "gate_bwd": 5 * B * T * C * s}
    dom = max(ms, key=lambda n: ms[n] * calls_per_step(n))
    achieved = nbytes[dom] / (ms[dom] * 1e-3) / 1e9
    ms_per_step = wall * 1e3 / args.steps
    res = {
        "metric": METRIC, "value": th / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name + "_block_scaffolding", "B": B, "T": T, "H": H, "dk": d, "C": C,
                   "pass": "fwd+bwd", "ops": "conv1d(k=4)+silu, rms qk-norm of q and k, silu gate",
                   "tokens_counted": "B*T*H"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_call": nbytes[dom],
                     "per_call_ms": ms,
                     "per_call_frac": {n: nbytes[n] / (ms[n] * 1e-3) / 1e9 / HBM_PEAK_GBS for n in ms}},
    }
    print(json.dumps(res), flush=True)


def bench_decode(args, dev, emit=True):
    """kla_decode_step (or kla_decode_step_pc) at the decode workload's shape, belief resident in HBM."""
    import torch
    import kla_inputs as K
    import paper_2602_10743_amd as kla
    w = K.WORKLOADS[4]
    S, H, dk, dv = w.B, w.H, w.dk, w.dv
    gen = torch.Generator(device=dev).manual_seed(0)
    steps_in = 8   # distinct per-step inputs, cycled
    n = lambda *sh: torch.randn(*sh, generator=gen, device=dev)
    sp = lambda *sh: torch.nn.functional.softplus(n(*sh))
    xs = []
    for _ in range(steps_in):
        k = n(S, H, dk)
        xs.append({"q": n(S, H, dk), "k": k / k.norm(dim=-1, keepdim=True), "v": n(S, H, dv),
                   "a": torch.sigmoid(n(S, H, dk) + 3.0), "p": sp(S, H, dk) * 0.05,
                   "r": sp(S, H, dv) if args.pc else sp(S, H)})
    lam = 1.0 + torch.rand((S, H, dk, dv) if args.pc else (S, H, dk), generator=gen, device=dev)
    eta = n(S, H, dk, dv)
    y = torch.empty((S, H, dv), device=dev)
    fn = kla.kla_decode_step_pc if args.pc else kla.kla_decode_step
    stream = torch.cuda.current_stream(dev)

    def step(i):
        x = xs[i % steps_in]
        fn(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], lam, eta, y=y)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(args.steps):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    # per (sequence, head): read and write the fp32 belief, read the fp32 inputs, write y
    belief = (2 * dk * dv if args.pc else dk * dv + dk)
    inputs = 4 * dk + dv + (dv if args.pc else 1)
    nbytes = S * H * (8 * belief + 4 * inputs + 4 * dv)
    achieved = nbytes / (ms * 1e-3) / 1e9
    res = {
        "metric": METRIC, "value": S * H / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name + ("_pc" if args.pc else ""), "S": S, "H": H, "dk": dk, "dv": dv,
                   "pass": "decode step", "tokens_counted": "S*H per step"},
        "roofline": {"bound": "hbm", "kernel": "kla_decode_step_pc" if args.pc else "kla_decode_step",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": None, "algorithmic_bytes_per_call": nbytes, "call_ms": ms},
    }
    if emit:
        print(json.dumps(res), flush=True)
    return res


def bench_a5(args, dev, emit=True):
    """kla_forward (saving the context) + kla_backward on the state-tracking workload (fp32).

    Its working set (~0.3 GB) is close to the 256 MB Infinity Cache, so a 1 GiB buffer is
    overwritten between the timed steps (outside the events) and every step starts from HBM;
    the per-step time is the mean of the event-timed steps."""
    import torch
    import kla_inputs as K
    import paper_2602_10743_amd as kla
    w = K.WORKLOADS[1]
    bits = K.full(w, as_bits=True)
    x = {n: torch.from_numpy(np.ascontiguousarray(bits[n])).to(dev) for n in bits}
    del bits
    stream = torch.cuda.current_stream(dev)
    if args.copy_calibration:
        from paper_2602_10743_amd.traffic import COPY_BYTES
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_state=False, save=True)
        if ev is not None:
            ev[1].record(stream)
        kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"],
                         saved=out["saved"], want_init_grads=False)
        if ev is not None:
            ev[2].record(stream)

    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for i in range(args.steps):
        flush.fill_(float(i))
        step(evs[i])
    torch.cuda.synchronize()
    del flush
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    bwd_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    wall = (fwd_ms + bwd_ms) * 1e-3 * args.steps
    th = w.token_heads
    fwd_b, bwd_b = algorithmic_bytes(w, 4)
    dom, ms, nbytes = ("kla_backward", bwd_ms, bwd_b * th) if bwd_ms >= fwd_ms else ("kla_forward", fwd_ms, fwd_b * th)
    achieved = nbytes / (ms * 1e-3) / 1e9
    from paper_2602_10743_amd.traffic import DIGEST_SOURCES_A5, load_summary
    measured = load_summary(os.path.join(ROOT, "profiles", "a5_state_tracking_traffic.md"), DIGEST_SOURCES_A5)
    res = {
        "metric": METRIC, "value": th / (wall / args.steps), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "T": w.T, "H": w.H, "dk": w.dk, "dv": w.dv, "pass": "fwd+bwd",
                   "tokens_counted": "B*T*H"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured.get(dom) if measured else None,
                     "traffic_unit": "bytes per call", "algorithmic_bytes_per_call": nbytes,
                     "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
                     "note": "chunked fp64 kernels (fp32 inputs, fp64 MFMA); Infinity Cache flushed between steps"},
    }
    if emit:
        print(json.dumps(res), flush=True)
    return res


def bench_long(args, dev, emit=True):
    """kla_forward (no saved context) on the long-context workload."""
    import torch
    import kla_inputs as K
    import paper_2602_10743_amd as kla
    w = K.WORKLOADS[3]
    bits = K.full(w, names=K.NAMES, as_bits=True)
    x = {n: torch.from_numpy(np.ascontiguousarray(bits[n].view(np.int16))).view(torch.bfloat16).to(dev)
         for n in bits}
    del bits
    stream = torch.cuda.current_stream(dev)
    y = torch.empty_like(x["v"])

    def step():
        kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_state=True, y=y)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = e0.elapsed_time(e1) / args.steps
    th = w.token_heads
    fwd_b, _ = algorithmic_bytes(w, 2)
    achieved = fwd_b * th / (ms * 1e-3) / 1e9
    res = {
        "metric": METRIC, "value": th / (wall / args.steps), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "T": w.T, "H": w.H, "dk": w.dk, "dv": w.dv, "pass": "fwd",
                   "tokens_counted": "B*T*H"},
        "roofline": {"bound": "hbm", "kernel": "kla_forward", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_call": fwd_b * th, "call_ms": ms},
    }
    if emit:
        print(json.dumps(res), flush=True)
    return res


def bench_mc(args, dev):
    """The Monte Carlo readout of KLA+ at the LM-layer shape with S = 10 draws: kla_mc_sample,
    its backward, and the logsumexp loss with its backward, inputs resident in HBM.  The
    draws (and their gradient, in the backward) are S copies of the bf16 readout, so the
    calls are priced on HBM bytes; the Philox rounds make the draw kernels VALU-heavy."""
    import torch
    import kla_inputs as K
    import paper_2602_10743_amd as kla
    w = K.WORKLOADS[2]
    B, T, H, dv, S, seed = w.B, w.T, w.H, w.dv, 10, 2026
    g = torch.Generator(device=dev).manual_seed(0)
    ymu = torch.randn((B, T, H, dv), generator=g, device=dev).to(torch.bfloat16)
    yvar = 0.05 + torch.rand((B, T, H), generator=g, device=dev)
    dys = torch.randn((S, B, T, H, dv), generator=g, device=dev).to(torch.bfloat16)
    n = B * T * H
    logp = -4.0 * torch.rand((S, n), generator=g, device=dev)
    dnll = torch.randn(n, generator=g, device=dev)
    stream = torch.cuda.current_stream(dev)
    names = ("kla_mc_sample", "kla_mc_sample_backward", "kla_mc_nll", "kla_mc_nll_backward")

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        kla.kla_mc_sample(ymu, yvar, S, seed)
        if ev is not None:
            ev[1].record(stream)
        kla.kla_mc_sample_backward(yvar, dys, seed)
        if ev is not None:
            ev[2].record(stream)
        kla.kla_mc_nll(logp)
        if ev is not None:
            ev[3].record(stream)
        kla.kla_mc_nll_backward(logp, dnll)
        if ev is not None:
            ev[4].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = [float(np.mean([e[k].elapsed_time(e[k + 1]) for e in evs])) for k in range(4)]
    el = B * T * H * dv
    # algorithmic bytes per call: read ymu, yvar, write S draws; read yvar, S gradients, write
    # dymu, dyvar; read logp, write nll; read logp, dnll, write dlogp
    nbytes = [2 * el + 4 * n + 2 * S * el, 4 * n + 2 * S * el + 2 * el + 4 * n, 4 * S * n + 4 * n,
              4 * S * n + 4 * n + 4 * S * n]
    calls = {nm: {"ms": m, "bytes": b, "hbm_frac": b / (m * 1e-3) / 1e9 / HBM_PEAK_GBS}
             for nm, m, b in zip(names, ms, nbytes)}
    dom = max(range(4), key=lambda k: ms[k])
    achieved = nbytes[dom] / (ms[dom] * 1e-3) / 1e9
    res = {
        "metric": METRIC, "value": n / (wall / args.steps), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name + "_mc", "B": B, "T": T, "H": H, "dv": dv, "S": S,
                   "pass": "draws + loss, forward and backward", "tokens_counted": "B*T*H"},
        "roofline": {"bound": "hbm", "kernel": names[dom], "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_call": nbytes[dom], "calls": calls},
    }
    print(json.dumps(res), flush=True)


def calls_per_step(name):
    return 2 if name.startswith("norm") else 1


def cpu_baseline(w, budget_s: float, ou=None):
    """fp64 oracle (forward + backward) on a few sampled (b, h) sequences.  With
    OU parameters ``ou`` the sample is every batch row of as many heads as fit
    (the parameters are per head), the oracle called once per head."""
    import kla_inputs as K
    import oracle
    threads = oracle.default_threads()
    n = max(1, min(4 * threads, w.B * w.H))
    if ou is None:
        pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
        g = np.random.default_rng(0)
        g.shuffle(pairs)
        groups = [sorted(pairs[:n])]
    else:
        groups = [[(b, h) for b in range(w.B)] for h in range(max(1, n // w.B))]
    tf = tb = 0.0
    count = 0
    for sample in groups:
        sl = K.pairs_slice(w, sample)
        t0 = time.perf_counter()
        if ou is None:
            oracle.forward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], nthreads=threads)
        else:
            h = sample[0][1]
            hp = {k: np.asarray(v[h:h + 1], dtype=np.float64) for k, v in ou.items()}
            oracle.forward_ou(sl["q"], sl["k"], sl["v"], hp["a"], hp["p"], hp["delta"], sl["r"], nthreads=threads)
        t1 = time.perf_counter()
        if ou is None:
            oracle.backward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], None, None, sl["dy"],
                            nthreads=threads)
        else:
            oracle.backward_ou(sl["q"], sl["k"], sl["v"], hp["a"], hp["p"], hp["delta"], sl["r"], None, None,
                               sl["dy"], nthreads=threads)
        t2 = time.perf_counter()
        tf += t1 - t0
        tb += t2 - t1
        count += len(sample)
    th = count * w.T
    return {"value": th / (tf + tb), "unit": "tokens/s", "cores": min(threads, max(len(s) for s in groups)),
            "kind": "oracle",
            "sample": f"{count} (batch, head) sequences of T={w.T} (fwd {tf:.1f}s + bwd {tb:.1f}s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="leave out the other workloads (state tracking, long context, decode)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain elementwise copy of known size first (counter calibration)")
    ap.add_argument("--ou", action="store_true",
                    help="OU gates: time-invariant (a, p, delta) instead of per-token abar, pbar")
    ap.add_argument("--pc", action="store_true",
                    help="per-channel-precision variant (elementwise scans), forward + backward")
    ap.add_argument("--decode", action="store_true",
                    help="decode step on the decode workload (with --pc: per-channel precision)")
    ap.add_argument("--long", action="store_true", help="forward of the long-context workload")
    ap.add_argument("--a5", action="store_true", help="fwd+bwd of the state-tracking workload (fp32)")
    ap.add_argument("--mc", action="store_true",
                    help="Monte Carlo readout (draws, logsumexp loss, their backward) at the LM-layer shape")
    ap.add_argument("--block", action="store_true",
                    help="block scaffolding around the layer (conv + SiLU, QK-norm, gate), forward + backward")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the filter layer shards over (batch, head) with no "
              "communication, and no multi-GPU path is implemented", file=sys.stderr)
        sys.exit(2)

    import torch
    import kla_inputs as K
    import paper_2602_10743_amd as kla

    w = K.WORKLOADS[2]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.decode:
        bench_decode(args, dev)
        return
    if args.long:
        bench_long(args, dev)
        return
    if args.a5:
        bench_a5(args, dev)
        return
    if args.mc:
        bench_mc(args, dev)
        return
    if args.pc:
        bench_pc(args, w, dev)
        return
    if args.block:
        bench_block(args, w, dev)
        return
    names = ("q", "k", "v", "r", "dy") if args.ou else K.NAMES + ("dy",)
    bits = K.full(w, names=names, as_bits=True)
    x = {n: torch.from_numpy(np.ascontiguousarray(bits[n].view(np.int16))).view(torch.bfloat16).to(dev)
         for n in bits}
    del bits
    ou_np = K.ou_params(w.H, w.dk, seed=w.cid) if args.ou else None
    ou = {n: torch.from_numpy(v).to(dev) for n, v in ou_np.items()} if args.ou else None
    stream = torch.cuda.current_stream(dev)
    if args.copy_calibration:
        from paper_2602_10743_amd.traffic import COPY_BYTES
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        if ou is None:
            out = kla.kla_forward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], want_state=False, save=True)
        else:
            out = kla.kla_forward_ou(x["q"], x["k"], x["v"], ou["a"], ou["p"], ou["delta"], x["r"],
                                     want_state=False, save=True)
        if ev is not None:
            ev[1].record(stream)
        if ou is None:
            kla.kla_backward(x["q"], x["k"], x["v"], x["a"], x["p"], x["r"], None, None, x["dy"],
                             saved=out["saved"], want_init_grads=False)
        else:
            kla.kla_backward_ou(x["q"], x["k"], x["v"], ou["a"], ou["p"], ou["delta"], x["r"], None, None,
                                x["dy"], saved=out["saved"], want_init_grads=False)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    bwd_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    ms_per_step = wall * 1e3 / args.steps
    th = w.token_heads
    fwd_b, bwd_b = algorithmic_bytes(w, 2, ou=args.ou)
    sfx = "_ou" if args.ou else ""
    if bwd_ms >= fwd_ms:
        dom, ms, nbytes = "kla_backward" + sfx, bwd_ms, bwd_b * th
    else:
        dom, ms, nbytes = "kla_forward" + sfx, fwd_ms, fwd_b * th
    achieved = nbytes / (ms * 1e-3) / 1e9
    from paper_2602_10743_amd.traffic import load_summary
    measured = load_summary(os.path.join(ROOT, "profiles", f"lm_layer{sfx}_traffic.md"))
    traffic = measured.get(dom) if measured else None
    res = {
        "metric": METRIC,
        "value": th / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name + sfx, "B": w.B, "T": w.T, "H": w.H, "dk": w.dk, "dv": w.dv,
                   "pass": "fwd+bwd", "gates": "ou (a, p, delta per head and key slot)" if args.ou else "per token",
                   "tokens_counted": "B*T*H"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_unit": "bytes per call", "algorithmic_bytes_per_call": nbytes,
                     "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
                     "algorithmic_bytes_per_token_head": {"fwd": fwd_b, "bwd": bwd_b}},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget, ou=ou_np)
    if not args.ou and not args.no_configs:
        del x
        torch.cuda.empty_cache()
        res["configs"] = other_configs(args, dev)
    print(json.dumps(res), flush=True)


def other_configs(args, dev):
    """The other workloads, each in its own pass and timing: the state-tracking fwd+bwd
    step (fp32, chunked fp64 kernels), the long-context forward and the decode step,
    with their HBM-roofline fractions on their algorithmic bytes."""
    import torch
    sub = argparse.Namespace(**vars(args))
    sub.pc = False
    out = {}
    for name, fn, steps in (("state_tracking_fwd_bwd", bench_a5, 20), ("long_context_fwd", bench_long, 5),
                            ("decode_step", bench_decode, 20)):
        sub.steps, sub.warmup = steps, 2
        r = fn(sub, dev, emit=False)
        rl = r["roofline"]
        out[name] = {"workload": r["config"]["workload"], "pass": r["config"]["pass"],
                     "ms": r["ms_per_step"], "value": r["value"], "unit": r["unit"], "dtype": r["dtype"],
                     "hbm_frac": rl["frac"], "kernel": rl["kernel"],
                     "algorithmic_bytes_per_call": rl["algorithmic_bytes_per_call"]}
        torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    main()
