"""Host sanitizer builds (CPU): the fp64 oracle and the C ABI layer, built with
AddressSanitizer and UndefinedBehaviorSanitizer by gcc / g++ and run by the drivers
under tests/asan/ (every oracle entry point on small shapes; every ABI path that
returns before device work, with its expected status)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def test_oracle_and_abi_under_sanitizers(tmp_path):
    if not shutil.which("gcc") or not shutil.which("g++"):
        pytest.skip("no host compiler")
    if not os.path.exists(os.path.join(ROOT, "paper_2602_10743_amd", "_build", "kla_api.o")):
        pytest.skip("library objects not built (paper_2602_10743_amd/build.py)")
    r = subprocess.run(["bash", os.path.join(HERE, "asan", "run.sh"), str(tmp_path)], capture_output=True,
                       text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "oracle sanitizer run: ok" in out and "ABI sanitizer run: ok" in out, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
