"""Host-side checks of bench.py and the traffic summaries (no GPU):

* more than one GPU is refused with a message, before torch is touched;
* the algorithmic bytes per token-head match the counts stated for the
  LM-layer workload (1538 B forward, 2820 B backward at d = 128, bf16; OU gates
  drop the per-token abar / pbar: 1026 and 1796 B);
* a traffic summary is used only while its source digest matches the sources
  of the measured kernels, and each workload's digest covers its own kernels.
"""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import kla_inputs as K  # noqa: E402
from paper_2602_10743_amd import traffic  # noqa: E402


def _bench_module():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_algorithmic_bytes_of_the_lm_layer():
    bench = _bench_module()
    w = K.WORKLOADS[2]
    assert (w.dk, w.dv, w.dtype) == (128, 128, "bf16")
    assert bench.algorithmic_bytes(w, 2) == (1538, 2820)
    assert bench.algorithmic_bytes(w, 2, ou=True) == (1026, 1796)


def _summary(digest, values):
    return "\n".join(["# test", f"sources: {digest}",
                      f"{traffic.SUMMARY_KEY}: " + ", ".join(f"{k}={v}" for k, v in values.items()), ""])


def test_traffic_summary_requires_matching_sources(tmp_path):
    vals = {"kla_forward": 1.5e8, "kla_backward": 2.5e8}
    good = tmp_path / "good.md"
    good.write_text(_summary(traffic.sources_digest(), vals))
    assert traffic.load_summary(str(good)) == vals
    stale = tmp_path / "stale.md"
    stale.write_text(_summary("0" * 64, vals))
    assert traffic.load_summary(str(stale)) is None
    assert traffic.load_summary(str(tmp_path / "missing.md")) is None
    # the state-tracking summary is checked against the token-recurrent sources
    a5 = tmp_path / "a5.md"
    a5.write_text(_summary(traffic.sources_digest(traffic.DIGEST_SOURCES_A5), vals))
    assert traffic.load_summary(str(a5), traffic.DIGEST_SOURCES_A5) == vals
    assert traffic.load_summary(str(a5)) is None


@pytest.mark.parametrize("names", [traffic.DIGEST_SOURCES, traffic.DIGEST_SOURCES_A5])
def test_digest_sources_exist(names):
    for name in names:
        assert os.path.exists(os.path.join(ROOT, "paper_2602_10743_amd", "csrc", name)), name
    assert "chunk64.hip" in traffic.DIGEST_SOURCES_A5 and "chunk64.hip" not in traffic.DIGEST_SOURCES


def test_digest_ignores_comments_only():
    a = "int f(int x) { // doubles\n  return 2 * x; /* twice */ }\n"
    b = "/* header */\nint f(int x) {\n    return 2 * x;\n}\n"
    assert traffic.code_text(a) == traffic.code_text(b)
    assert traffic.code_text(a) != traffic.code_text(a.replace("2 * x", "3 * x"))


def test_trace_table_from_kernel_stats(tmp_path):
    stats = tmp_path / "bench_kernel_stats.csv"
    stats.write_text(
        '"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n'
        '"void kla::(anonymous namespace)::bwd_dk_kernel<128, 128, false, false>(kla::Shape, kla::BwdArgs)",'
        '"2","900000","450000","60.0","440000","460000","1"\n'
        '"void kla::(anonymous namespace)::fwd_chunk_kernel<128, 128, false, false, false>(kla::Shape)",'
        '"2","600000","300000","40.0","290000","310000","1"\n'
        '"at::native::fill_kernel(float)","5","100","20","0.0","10","30","1"\n')
    out = traffic.trace_table(str(stats), ["bwd_dk", "fwd_chunk"]).splitlines()
    assert out[0].startswith("| kernel | calls | avg us")
    assert out[2] == "| bwd_dk_kernel<128, 128, false, false> | 2 | 450.0 | 440.0 | 460.0 | 60.0% |"
    assert out[3] == "| fwd_chunk_kernel<128, 128, false, false, false> | 2 | 300.0 | 290.0 | 310.0 | 40.0% |"
    assert len(out) == 4   # the fill kernel is left out
