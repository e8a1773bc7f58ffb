"""The cross-stream ordering of ring launches (csrc/ring_gate.h), tested on
the host with a fake stream API under ThreadSanitizer (no GPU): launches on
one stream are not ordered further, a launch on another stream waits for
the previous ring launch, captured launches are left alone, devices are
independent, API errors stop the launch, and concurrent launchers never let
two ring launches overlap."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_ring_gate_under_tsan(tmp_path):
    if not shutil.which("g++"):
        pytest.skip("g++ not available")
    exe = str(tmp_path / "ring_gate_test")
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-pthread", "-fsanitize=thread", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "paper_2603_11438_amd", "csrc"),
           os.path.join(ROOT, "tests", "native", "ring_gate_test.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, TSAN_OPTIONS="halt_on_error=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ring gate: ok" in r.stdout
    assert "WARNING: ThreadSanitizer" not in r.stderr
