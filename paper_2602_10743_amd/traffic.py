"""HBM traffic of the KLA calls from two rocprofv3 counter runs of bench.py.

FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are collected in separate runs,
each over a bench run with --copy-calibration, which adds a plain elementwise
copy of COPY_BYTES (read) + COPY_BYTES (written).  The counters of that copy
kernel give the scale from counter units to bytes; the scaled counters of the
kernels of one forward call and one backward call are the measured traffic.
The summary records a digest of the kernel sources; bench.py reports the
traffic only while the sources still match it.

Run from the repository root on the GPU machine (TMPDIR=/tmp):
  rocprofv3 --pmc FETCH_SIZE --output-format csv -d D/fetch -o run -- \\
      python bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-configs --copy-calibration
  rocprofv3 --pmc WRITE_SIZE --output-format csv -d D/write -o run -- \\
      python bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-configs --copy-calibration
  python -m paper_2602_10743_amd.traffic D/fetch D/write > profiles/lm_layer_traffic.md

With OU gates: the same two runs with `bench.py ... --ou`, then
  python -m paper_2602_10743_amd.traffic D/fetch D/write --ou > profiles/lm_layer_ou_traffic.md

The state-tracking workload (fp32, chunked fp64 kernels): the same two runs with
`bench.py --a5 --steps 2 --warmup 1 --copy-calibration`, then
  python -m paper_2602_10743_amd.traffic D/fetch D/write --a5 > profiles/a5_state_tracking_traffic.md

The kernel-trace tables of profiles/*_kernel_trace.md come from the stats file of a
`rocprofv3 --kernel-trace --stats --output-format csv -d D/trace -o bench -- python bench.py ...`
run:
  python -m paper_2602_10743_amd.traffic --trace D/trace/bench_kernel_stats.csv [name,name,...]
(the optional list keeps the kernels whose names contain one of the given parts).

MFMA and VALU utilisation per kernel come from a third run:
  rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU \\
      GRBM_GUI_ACTIVE --output-format csv -d D/util -o run -- \\
      python bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-configs
  python -m paper_2602_10743_amd.traffic --util D/util > profiles/lm_layer_mfma_valu.md
"""
import csv
import glob
import hashlib
import os
import re
import sys
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
COPY_BYTES = 256 << 20
CALLS = {
    "kla_forward": ("fwd_chunk_kernel",),
    "kla_backward": ("bwd_dv_kernel", "bwd_dk_kernel", "dr_combine_kernel"),
}
CALLS_OU = {
    "kla_forward_ou": ("fwd_chunk_kernel",),
    "kla_backward_ou": ("bwd_dv_kernel", "bwd_dk_kernel", "dr_combine_kernel", "ou_param_grads_kernel"),
}
CALLS_A5 = {
    "kla_forward": ("fwd64_kernel",),
    "kla_backward": ("bwd64_kernel",),
}
SUMMARY_KEY = "traffic_bytes_per_call"


# the sources the measured calls are built from: the ABI layer, the shared
# headers and the chunked kernels (and the OU parameter gradients)
DIGEST_SOURCES = ("kla_api.cpp", "kla_internal.hpp", "kla_device.hpp", "kla_buf.hpp", "kla_mfma.hpp",
                  "kla_chunk.hpp", "chunk_fwd.hip", "chunk_bwd_dv.hip", "chunk_bwd_dk.hip", "ou.hip",
                  "validate.hip")
# ... and of the token-recurrent kernels (the state-tracking workload)
DIGEST_SOURCES_A5 = ("kla_api.cpp", "kla_internal.hpp", "kla_device.hpp", "kla_buf.hpp", "chunk64.hip",
                     "validate.hip")


def code_text(text: str) -> str:
    """The source without its comments and with whitespace runs collapsed, so
    that an edit of comments alone leaves the digest as it was (the sources
    hold no comment markers inside string literals)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def sources_digest(names=DIGEST_SOURCES) -> str:
    """sha256 over the code (comments stripped) of the measured kernels'
    sources, in name order."""
    h = hashlib.sha256()
    for name in sorted(names):
        h.update(name.encode())
        with open(os.path.join(HERE, "csrc", name), encoding="utf-8") as f:
            h.update(code_text(f.read()).encode())
    return h.hexdigest()


def _short(name: str) -> str:
    return re.sub(r"\(.*", "", name.replace("void ", "").replace("kla::(anonymous namespace)::", ""))


def _counter(run_dir: str, counter: str) -> dict:
    """kernel short name -> list of per-dispatch counter values."""
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    vals = defaultdict(dict)
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            key = (r.get("Dispatch_Id") or r.get("Correlation_Id"), _short(r["Kernel_Name"]))
            vals[key[1]][key[0]] = vals[key[1]].get(key[0], 0.0) + float(r["Counter_Value"])
    return {k: list(v.values()) for k, v in vals.items()}


def _per_call(vals: dict, scale: float, calls: dict) -> dict:
    out = {}
    for call, kernels in calls.items():
        total = 0.0
        for kname in kernels:
            hits = [v for k, v in vals.items() if k.startswith(kname)]
            if not hits:
                raise KeyError(f"kernel {kname} not in the counter run")
            seq = hits[0]
            total += sum(seq) / len(seq) * scale
        out[call] = total
    return out


def summarise(fetch_dir: str, write_dir: str, ou: bool = False, a5: bool = False) -> str:
    calls = CALLS_A5 if a5 else CALLS_OU if ou else CALLS
    flag = " --a5" if a5 else " --ou" if ou else ""
    names = DIGEST_SOURCES_A5 if a5 else DIGEST_SOURCES
    fetch = _counter(fetch_dir, "FETCH_SIZE")
    write = _counter(write_dir, "WRITE_SIZE")
    kla_names = tuple(k for ks in calls.values() for k in ks)
    copies = [k for k in fetch if not k.startswith(kla_names)]
    if not copies:
        raise KeyError("no calibration copy kernel in the fetch run")
    copy = max(copies, key=lambda k: max(fetch[k]))
    f_fetch = COPY_BYTES / max(fetch[copy])          # bytes per counter unit
    f_write = COPY_BYTES / max(write[copy])
    rd = _per_call(fetch, f_fetch, calls)
    wr = _per_call(write, f_write, calls)
    title = ("state-tracking workload (B=64, T=512, H=4, d=32, fp32)" if a5 else
             "lm-layer workload (B=8, T=2048, H=16, d=128, bf16" + (", OU gates)" if ou else ")"))
    lines = [
        "# HBM traffic per call, " + title,
        "",
        "Counters: FETCH_SIZE and WRITE_SIZE from two separate `rocprofv3 --pmc` runs of",
        ("`python bench.py --a5 --steps 2 --warmup 1 --copy-calibration`, scaled by" if a5 else
         f"`python bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-configs --copy-calibration{flag}`, scaled by"),
        f"the calibration copy kernel `{copy}` ({COPY_BYTES} bytes read and written):",
        f"fetch scale {f_fetch:.4f} bytes/unit, write scale {f_write:.4f} bytes/unit.",
        "",
        "| call | read bytes | written bytes | total |",
        "|---|---|---|---|",
    ]
    for call in calls:
        lines.append(f"| {call} | {rd[call]:.4g} | {wr[call]:.4g} | {rd[call] + wr[call]:.4g} |")
    lines += [
        "",
        f"sources: {sources_digest(names)}",
        f"{SUMMARY_KEY}: " + ", ".join(f"{c}={rd[c] + wr[c]:.6g}" for c in calls),
        "",
    ]
    return "\n".join(lines)


def load_summary(path: str, names=DIGEST_SOURCES):
    """{call: bytes} from a summary written by summarise(), or None when the file
    is missing or was taken from different kernel sources (names: the digest's sources)."""
    if not os.path.exists(path):
        return None
    digest, values = None, None
    for line in open(path):
        if line.startswith("sources: "):
            digest = line.split(":", 1)[1].strip()
        elif line.startswith(SUMMARY_KEY + ": "):
            values = {}
            for item in line.split(":", 1)[1].split(","):
                k, v = item.strip().split("=")
                values[k] = float(v)
    if digest != sources_digest(names) or values is None:
        return None
    return values


UTIL_COUNTERS = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU", "GRBM_GUI_ACTIVE")
# the state-tracking workload (fp32 inputs) runs fp64 MFMAs
UTIL_COUNTERS_A5 = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_F64", "SQ_INSTS_VALU", "GRBM_GUI_ACTIVE")
F64_PEAK = 78.6e12       # fp64 flop/s (matrix and vector alike)
NUM_SIMD = 1024          # 256 CUs x 4 SIMDs
NUM_XCD = 8              # GRBM_GUI_ACTIVE comes summed over the accelerator dies
BF16_PEAK = 2.5e15       # dense bf16 MFMA flop/s
VALU_PEAK_INSTS = 256 * 4 * 2.4e9 / 4   # wave64 VALU instructions per second (one per 4 cycles per SIMD)


def _rows(run_dir: str):
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    for f in files:
        yield from csv.DictReader(open(f))


def summarise_util(run_dir: str, a5: bool = False) -> str:
    """MFMA busy fraction, MFMA flop rate (bf16; fp64 for the state-tracking
    workload) and VALU issue per kernel from one counter run with UTIL_COUNTERS
    (UTIL_COUNTERS_A5); durations from the dispatch timestamps."""
    acc = defaultdict(lambda: defaultdict(float))   # kernel -> counter -> sum over dispatches
    dur = defaultdict(dict)                          # kernel -> dispatch -> ns
    tables = [CALLS_A5] if a5 else [CALLS, CALLS_OU]
    for r in _rows(run_dir):
        k = _short(r["Kernel_Name"])
        if not k.startswith(tuple(n for t in tables for ns in t.values() for n in ns)):
            continue
        d = r.get("Dispatch_Id") or r.get("Correlation_Id")
        acc[k][r["Counter_Name"]] += float(r["Counter_Value"])
        dur[k][d] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    mops, peak, kind = (("SQ_INSTS_VALU_MFMA_MOPS_F64", F64_PEAK, "fp64") if a5 else
                        ("SQ_INSTS_VALU_MFMA_MOPS_BF16", BF16_PEAK, "bf16"))
    title = ("state-tracking workload (B=64, T=512, H=4, d=32, fp32 inputs, fp64 arithmetic)" if a5 else
             "lm-layer workload (B=8, T=2048, H=16, d=128, bf16)")
    cmd = ("python bench.py --a5 --steps 2 --warmup 1 --no-cpu-baseline" if a5 else
           "python bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-configs")
    lines = [
        f"# MFMA and VALU utilisation per kernel, {title}",
        "",
        "Command (repository root, one MI355X, TMPDIR=/tmp):",
        "",
        "    rocprofv3 --pmc " + " ".join(UTIL_COUNTERS_A5 if a5 else UTIL_COUNTERS) +
        " --output-format csv -d D/util -o run -- " + cmd,
        "    python -m paper_2602_10743_amd.traffic " + ("--util-a5" if a5 else "--util") + " D/util",
        "",
        "Durations come from the dispatch timestamps of the same run.  MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / ",
        f"{NUM_XCD} dies x {NUM_SIMD} SIMDs); {kind} rate = 512 x {mops} / duration against",
        f"{peak / 1e12:.1f} TFLOP/s; VALU issue = SQ_INSTS_VALU / duration against one wave64",
        "instruction per 4 cycles per SIMD at 2.4 GHz." + ("" if a5 else "  The split-bf16 products count 2-3 MFMAs"),
    ]
    if not a5:
        lines.append("per fp32-accurate product.")
    lines += [
        "",
        f"| kernel | dispatches | avg us | MFMA busy | {kind} MFMA TFLOP/s | of peak | VALU Ginst/s | of peak |",
        "|---|---|---|---|---|---|---|---|",
    ]
    for k in sorted(acc):
        n = len(dur[k])
        t = sum(dur[k].values()) / n * 1e-9
        c = {name: v / n for name, v in acc[k].items()}
        active = c.get("GRBM_GUI_ACTIVE", 1.0) / NUM_XCD
        busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / max(active * NUM_SIMD, 1.0)
        flops = 512.0 * c.get(mops, 0.0) / t
        valu = c.get("SQ_INSTS_VALU", 0.0) / t
        lines.append(f"| {k} | {n} | {t * 1e6:.1f} | {100 * busy:.1f}% | {flops / 1e12:.1f} | "
                     f"{100 * flops / peak:.1f}% | {valu / 1e9:.1f} | {100 * valu / VALU_PEAK_INSTS:.1f}% |")
    lines.append("")
    return "\n".join(lines)


def trace_table(stats_csv: str, keep=None) -> str:
    """Markdown table of a rocprofv3 kernel_stats.csv: calls, average, min and max
    duration (us) and share of the total, longest first."""
    rows = []
    with open(stats_csv, newline="") as f:
        for r in csv.DictReader(f):
            name = re.sub(r"\(.*\)$", "", r["Name"].replace("void ", "").replace("kla::(anonymous namespace)::", ""))
            if keep and not any(k in name for k in keep):
                continue
            rows.append((name, int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                         float(r["MaxNs"]) / 1e3, float(r["TotalDurationNs"])))
    total = sum(r[5] for r in rows) or 1.0
    rows.sort(key=lambda r: -r[5])
    out = ["| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for name, calls, avg, lo, hi, tot in rows:
        out.append(f"| {name} | {calls} | {avg:.1f} | {lo:.1f} | {hi:.1f} | {100 * tot / total:.1f}% |")
    return "\n".join(out)


if __name__ == "__main__":
    if len(sys.argv) in (3, 4) and sys.argv[1] == "--trace":
        print(trace_table(sys.argv[2], sys.argv[3].split(",") if len(sys.argv) == 4 else None))
        sys.exit(0)
    if len(sys.argv) == 3 and sys.argv[1] in ("--util", "--util-a5"):
        print(summarise_util(sys.argv[2], a5=sys.argv[1] == "--util-a5"))
        sys.exit(0)
    ou = "--ou" in sys.argv[1:]
    a5 = "--a5" in sys.argv[1:]
    args = [a for a in sys.argv[1:] if a not in ("--ou", "--a5")]
    if len(args) != 2:
        print(__doc__, file=sys.stderr)
        sys.exit(2)
    print(summarise(args[0], args[1], ou=ou, a5=a5))
