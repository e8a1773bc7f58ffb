"""Profiler -> tuner closed loop (host side, no GPU): the telemetry map and
the adaptive channel tuner, driven with synthetic latencies in the paper's
three phases (section 5.3, composability): baseline, a 10x latency spike,
recovery."""
from __future__ import annotations

import ctypes
import os
import subprocess

import pytest

import paper_2603_11438_amd as ar

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(autouse=True)
def clean():
    ar.lib()
    ar.ar_profile_clear()
    yield
    ar.ar_set_tuner(None)
    ar.ar_profile_clear()


def test_lookup_is_null_checked():
    assert ar.ar_profile_lookup(12345) is None
    ar.ar_profile_record(12345, 987654, 7)
    st = ar.ar_profile_lookup(12345)
    assert st == {"comm_id": 12345, "latency_ns": 987654, "nchannels": 7, "samples": 1}
    ar.ar_profile_record(12345, 5, 3)
    assert ar.ar_profile_lookup(12345)["samples"] == 2
    assert ar.ar_profile_lookup(12346) is None
    with pytest.raises(ar.ARError):
        ar.ar_profile_record(1, 1, 70000)


def test_map_capacity_is_fixed():
    for i in range(1024):
        ar.ar_profile_record(10_000 + i, i, 1)
    with pytest.raises(ar.ARError) as ei:
        ar.ar_profile_record(99_999, 1, 1)
    assert ei.value.code == ar.AR_ERR_NOMEM


def _latency(ch, contended):
    # A synthetic run latency that falls with more channels.
    base = 100_000 * 12 // ch
    return base * 10 if contended else base


def _phase(comm, calls, contended, record=True):
    L = ar.lib()
    ctx = ar.ar_tune_ctx(ar.AR_COLL_ALLREDUCE, 64 << 20, 8, ar.AR_FLOAT32, 64, comm)
    out = ar.ar_tune_out()
    trace = []
    for _ in range(calls):
        assert L.ar_tune(ctypes.byref(ctx), ctypes.byref(out)) == ar.AR_OK
        trace.append(out.nchannels)
        if record:
            assert L.ar_profile_record(comm, _latency(out.nchannels, contended), out.nchannels) == ar.AR_OK
    return trace


def test_adaptive_without_profiler_stays_at_two():
    ar.ar_set_tuner("adaptive")
    trace = _phase(7, 20000, False, record=False)
    assert set(trace) == {2}


def test_adaptive_three_phases():
    ar.ar_set_tuner("adaptive")
    comm = 42
    p1 = _phase(comm, 100_000, False)
    assert p1[0] == 2 and p1[-1] == 12
    assert all(b >= a for a, b in zip(p1, p1[1:]))          # monotone ramp
    assert p1.index(12) <= 100_000
    p2 = _phase(comm, 100_000, True)                        # 10x latency spike
    assert p2[2] == 2 and set(p2[2:]) == {2}                # backs off at once, stays down
    p3 = _phase(comm, 100_000, False)                       # recovery
    assert p3[-1] == 12 and p3.index(12) <= 100_000
    assert all(b >= a for a, b in zip(p3, p3[1:]))


def test_adaptive_config_and_invalid_config():
    ar.ar_set_tuner("adaptive", adaptive={"min_channels": 3, "max_channels": 5, "ramp_calls": 10})
    trace = _phase(9, 100, False)
    assert trace[0] == 3 and max(trace) == 5
    # an invalid configuration makes the tuner fail, so decisions fall back
    ar.ar_set_tuner("adaptive", adaptive={"min_channels": 0})
    assert ar.ar_tune(1 << 20, comm_id=9)["nchannels"] == 16


def test_telemetry_concurrent_under_tsan(tmp_path):
    exe = str(tmp_path / "telemetry_race")
    src = os.path.join(ROOT, "tests", "native", "telemetry_race.cpp")
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-pthread", "-fsanitize=thread", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2603_11438_amd", "csrc"), src,
           os.path.join(ROOT, "paper_2603_11438_amd", "csrc", "ar_profile.cpp"),
           os.path.join(ROOT, "paper_2603_11438_amd", "csrc", "ar_tuner.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, TSAN_OPTIONS="halt_on_error=1"))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "WARNING: ThreadSanitizer" not in r.stderr


def test_listing1_policy():
    """The paper's Listing 1 rules over the shared telemetry."""
    ar.ar_set_tuner("size_adaptive")
    # no map entry: the listing sets 4 channels and returns, leaving the
    # algorithm and protocol to the library's default (the Simple ring)
    raw = ar.ar_tuner_raw("size_adaptive", 32 * 1024, comm_id=5)
    assert (raw["nchannels"], raw["algo"], raw["proto"]) == (4, ar.AR_ALGO_AUTO, ar.AR_PROTO_AUTO)
    for size in (4096, 32 * 1024, 1 << 20):
        d = ar.ar_tune(size, comm_id=5)
        assert (d["nchannels"], d["algo"], d["proto"]) == (4, ar.AR_ALGO_RING, ar.AR_PROTO_SIMPLE)
    # with a sample the size threshold picks the algorithm, with Simple
    ar.ar_profile_record(5, 500_000, 6)
    d = ar.ar_tune(32 * 1024, comm_id=5)
    assert (d["nchannels"], d["algo"], d["proto"]) == (6, ar.AR_ALGO_DIRECT, ar.AR_PROTO_SIMPLE)
    d = ar.ar_tune(32 * 1024 + 1, comm_id=5)
    assert (d["nchannels"], d["algo"], d["proto"]) == (6, ar.AR_ALGO_RING, ar.AR_PROTO_SIMPLE)
    # fast runs keep the recorded channel count
    assert ar.ar_tune(1 << 20, comm_id=5)["nchannels"] == 6
    # slow runs (> 1 ms) add a channel, up to 16
    ar.ar_profile_record(5, 2_000_000, 6)
    assert ar.ar_tune(1 << 20, comm_id=5)["nchannels"] == 7
    ar.ar_profile_record(5, 2_000_000, 16)
    assert ar.ar_tune(1 << 20, comm_id=5)["nchannels"] == 16
    # the closed loop converges upward under sustained slowness
    ch = 4
    for _ in range(20):
        ar.ar_profile_record(8, 5_000_000, ch)
        ch = ar.ar_tune(1 << 24, comm_id=8)["nchannels"]
    assert ch == 16
