"""CPU: the HIP-free host layer (page pool, conversation table, work plans, placement) built with
g++ -fsanitize=address,undefined and run."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_01839_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_metadata_under_sanitizers():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "test_host")
        cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=all", "-I", CSRC,
               os.path.join(ROOT, "tests", "cpp", "test_host.cpp"),
               os.path.join(CSRC, "host", "host_state.cpp"), os.path.join(CSRC, "host", "sched.cpp"),
               "-o", exe]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        r = subprocess.run([exe], capture_output=True, text=True, timeout=120,
                           env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"})
        assert r.returncode == 0, r.stdout + r.stderr
        assert "passed" in r.stdout
