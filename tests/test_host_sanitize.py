"""The library's host builder (api.cpp: validation, routing, workload
expansion, engine choice and table construction, everything before the
first device call) under AddressSanitizer and UndefinedBehaviorSanitizer.
It is built host-only with g++ against a stand-in HIP header that has no
device (tests/hip_host_stub), loaded into a Python process with the ASan
runtime preloaded, and driven by tests/host_sanitize_drive.py over the
mixed-feature fuzz workloads and the benchmark configurations."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_builder_under_sanitizers(tmp_path):
    lib = tmp_path / "libsimgpu_host.so"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fPIC", "-shared",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-I", os.path.join(HERE, "hip_host_stub"), "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2606_10440_amd", "csrc", "api.cpp"),
           os.path.join(HERE, "hip_host_stub", "engines_stub.cpp"), "-o", str(lib)]
    subprocess.run(cmd, check=True)
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    env = dict(os.environ, LD_PRELOAD=asan, SIMGPU_LIB=str(lib), PYTHONPATH=ROOT,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("SIMGPU_ENGINE", None)
    r = subprocess.run([sys.executable, os.path.join(HERE, "host_sanitize_drive.py")], capture_output=True,
                       text=True, env=env, timeout=900)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-6000:]
    assert "workloads ok" in r.stdout and "runtime error" not in r.stderr, r.stderr[-6000:]
