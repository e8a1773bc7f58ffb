"""Host-code checks of libar's tuner and geometry built with g++ under
sanitizers (no GPU): the hot-reload concurrency test under
ThreadSanitizer and a randomised geometry/tuner check under
AddressSanitizer + UndefinedBehaviorSanitizer, plus the Python-facing
reload semantics."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

import paper_2603_11438_amd as ar

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
TUNER_SRC = os.path.join(ROOT, "paper_2603_11438_amd", "csrc", "ar_tuner.cpp")
INCS = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2603_11438_amd", "csrc")]


def _build(tmp_path, src, sanitize):
    if not shutil.which("g++"):
        pytest.skip("g++ not available")
    exe = str(tmp_path / os.path.splitext(os.path.basename(src))[0])
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-pthread", f"-fsanitize={sanitize}", "-fno-omit-frame-pointer",
           *INCS, os.path.join(NATIVE, src), TUNER_SRC, "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def test_hot_reload_concurrent_under_tsan(tmp_path):
    exe = _build(tmp_path, "tuner_reload_test.cpp", "thread")
    r = subprocess.run([exe, "400000", "4"], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, TSAN_OPTIONS="halt_on_error=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "calls 400000 bad 0 torn 0 after_retire 0" in r.stdout, r.stdout
    assert "WARNING: ThreadSanitizer" not in r.stderr


def test_geometry_fuzz_under_asan_ubsan(tmp_path):
    exe = _build(tmp_path, "geometry_fuzz.cpp", "address,undefined")
    r = subprocess.run([exe, "200000"], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, UBSAN_OPTIONS="halt_on_error=1", ASAN_OPTIONS="detect_leaks=0"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "failures 0" in r.stdout


def test_reload_rejects_malformed_and_keeps_old():
    ar.lib()
    ar.ar_set_tuner(lambda ctx: {"proto": ar.AR_PROTO_LL, "nchannels": 5})
    before = ar.ar_tune(1 << 20)
    with pytest.raises(ar.ARError) as ei:
        ar.ar_reload_tuner(lambda ctx: {"proto": 42, "nchannels": 1})
    assert ei.value.code == ar.AR_ERR_ARG
    assert ar.ar_tune(1 << 20) == before
    # a tuner that fails only on some contexts is caught by the probe grid
    with pytest.raises(ar.ARError):
        ar.ar_reload_tuner(lambda ctx: {"proto": ar.AR_PROTO_SIMPLE, "rc": 1 if ctx["nranks"] == 16 else 0})
    assert ar.ar_tune(1 << 20) == before
    # a well-formed but poor policy (one channel everywhere) is accepted
    st = ar.ar_reload_tuner(lambda ctx: {"proto": ar.AR_PROTO_SIMPLE, "nchannels": 1})
    assert st["probes"] > 100 and st["swap_ns"] < 10_000_000
    assert ar.ar_tune(1 << 20)["nchannels"] == 1
    ar.ar_set_tuner(None)


def test_decision_latency_native(tmp_path):
    """1 M host decisions: reported for context beside the paper's figures."""
    exe = str(tmp_path / "tune_latency")
    subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", *INCS, os.path.join(NATIVE, "tune_latency.cpp"),
                    TUNER_SRC, "-o", exe], check=True, capture_output=True)
    r = subprocess.run([exe, "1000000"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0
    print(r.stdout)
    p50 = int(r.stdout.split("p50 ")[1].split()[0])
    assert p50 < 2000
