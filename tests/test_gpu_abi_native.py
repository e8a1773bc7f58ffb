"""The C ABI without Python in the loop: a host program (built by the build
step from tests/native/abi_gpu_check.cpp) allocates rank buffers with
hipMalloc and plans and runs AllReduces through libar's exported calls
only, checking every element against exact integer sums."""
from __future__ import annotations

import os
import subprocess

import pytest

from tests.gpu_helpers import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "native", "abi_gpu_check")


def test_c_abi_from_a_native_program():
    assert os.path.exists(EXE), "tests/native/abi_gpu_check is not built: run __graft_entry__.build()"
    say("native C-ABI check")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert r.stdout.strip().endswith("abi gpu check: ok"), r.stdout[-3000:]
