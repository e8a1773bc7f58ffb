"""The build entry point compiles the library and the C oracle from source
and accepts what it built (run in a child process, as a build driver would)."""
from __future__ import annotations

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_build_entry_point_succeeds():
    r = subprocess.run([sys.executable, "-c", "import __graft_entry__ as g; g.build(); print('built')"],
                       cwd=ROOT, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.strip().endswith("built")
    # the host program that drives the C ABI alone is built too
    assert os.access(os.path.join(ROOT, "tests", "native", "abi_gpu_check"), os.X_OK)
