"""The library's host logic under AddressSanitizer (CPU): plans and index
maps, the collector, workspace carving and table uploads of every entry
point, the allocation-free call and the error paths, run against a stand-in
HIP runtime whose "device" buffers are exact-size host allocations
(tests/asan/host_checks.cpp, tests/asan/build_and_run.py)."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(not os.path.exists("/opt/rocm/llvm/bin/clang++"), reason="needs the ROCm clang")
def test_host_code_is_clean_under_asan(tmp_path):
    r = subprocess.run([sys.executable, os.path.join(HERE, "asan", "build_and_run.py"), str(tmp_path)],
                       capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "host checks ok" in r.stdout
    assert "AddressSanitizer" not in r.stderr and "LeakSanitizer" not in r.stderr
