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


def algorithmic_bytes(w, s):
    """Per token-head: forward reads q,k,abar,pbar (dk each), v (dv), r (1) and
    writes y (dv); backward reads those plus dy and writes the six gradients."""
    fwd = (4 * w.dk + w.dv + 1) * s + w.dv * s
    bwd = 2 * (4 * w.dk + w.dv + 1) * s + w.dv * s
    return fwd, bwd


def cpu_baseline(w, budget_s: float):
    """fp64 oracle (forward + backward) on a few sampled (b, h) sequences."""
    import kla_inputs as K
    import oracle
    threads = oracle.default_threads()
    pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
    g = np.random.default_rng(0)
    g.shuffle(pairs)
    n = max(1, min(4 * threads, len(pairs)))
    sample = sorted(pairs[:n])
    sl = K.pairs_slice(w, sample)
    t0 = time.perf_counter()
    oracle.forward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], nthreads=threads)
    t1 = time.perf_counter()
    oracle.backward(sl["q"], sl["k"], sl["v"], sl["a"], sl["p"], sl["r"], None, None, sl["dy"], nthreads=threads)
    t2 = time.perf_counter()
    th = len(sample) * w.T
    return {"value": th / (t2 - t0), "unit": "tokens/s", "cores": min(threads, len(sample)), "kind": "oracle",
            "sample": f"{len(sample)} (batch, head) sequences of T={w.T} (fwd {t1 - t0:.1f}s + bwd {t2 - t1:.1f}s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain elementwise copy of known size first (counter calibration)")
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
    bits = K.full(w, as_bits=True)
    x = {n: torch.from_numpy(np.ascontiguousarray(bits[n].view(np.int16))).view(torch.bfloat16).to(dev)
         for n in bits}
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
    fwd_b, bwd_b = algorithmic_bytes(w, 2)
    if bwd_ms >= fwd_ms:
        dom, ms, nbytes = "kla_backward", bwd_ms, bwd_b * th
    else:
        dom, ms, nbytes = "kla_forward", fwd_ms, fwd_b * th
    achieved = nbytes / (ms * 1e-3) / 1e9
    from paper_2602_10743_amd.traffic import load_summary
    measured = load_summary(os.path.join(ROOT, "profiles", "lm_layer_traffic.md"))
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
        "config": {"workload": w.name, "B": w.B, "T": w.T, "H": w.H, "dk": w.dk, "dv": w.dv,
                   "pass": "fwd+bwd", "tokens_counted": "B*T*H"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_unit": "bytes per call", "algorithmic_bytes_per_call": nbytes,
                     "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
                     "algorithmic_bytes_per_token_head": {"fwd": fwd_b, "bwd": bwd_b}},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
