"""Host-side checks of libar that need no GPU: the library loads and exports
every entry point include/ar.h declares; the tuner validates, clamps and
falls back; the plan geometry matches the oracle's segment rule; the
bus-bandwidth formula matches the paper's own pair of numbers."""
from __future__ import annotations

import ctypes
import os
import re
import time

import numpy as np
import pytest

import paper_2603_11438_amd as ar
from oracle import ring_oracle as ro

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ar.h")


@pytest.fixture(scope="module", autouse=True)
def built_lib():
    if not os.path.exists(ar.LIB_PATH):
        import __graft_entry__

        __graft_entry__.build()
    ar.lib()
    yield
    ar.ar_set_tuner(None)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = set(re.findall(r"\b(ar_[a-z0-9_]+)\s*\(", text))
    # typedef'd function pointer type is not a symbol
    names.discard("ar_tuner_fn")
    return sorted(names)


def test_every_declared_symbol_is_exported():
    names = header_functions()
    assert len(names) >= 20
    L = ctypes.CDLL(ar.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    # and the binding covers the same set
    assert set(names) == set(ar.SIGNATURES), set(names) ^ set(ar.SIGNATURES)


def test_version_and_strerror():
    with open(os.path.join(ROOT, "include", "ar.h")) as f:
        hdr = int(re.search(r"#define AR_VERSION (\d+)", f.read()).group(1))
    assert ar.ar_version() == ar.AR_VERSION == hdr == 4
    for code in range(9):
        assert ar.ar_strerror(code) != "unknown error", code
    assert ar.ar_strerror(99) == "unknown error"


# ------------------------------------------------------------------ tuner

@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_builtin_table_form(dtype):
    # one decision per power-of-two bucket, small sizes latency-oriented;
    # AllReduce has a table per data type (bf16 hops carry fp32 partials)
    prev = None
    for k in range(12, 28):
        d = ar.ar_tune(1 << k, dtype=dtype)
        assert d["proto"] in (ar.AR_PROTO_LL, ar.AR_PROTO_LL128, ar.AR_PROTO_SIMPLE)
        assert 1 <= d["nchannels"] <= ar.AR_MAX_CHANNELS
        assert d["chunk_bytes"] >= 16 and d["chunk_bytes"] % 16 == 0
        assert 1 <= d["nwaves"] <= ar.AR_MAX_WAVES
        assert d["algo"] in (ar.AR_ALGO_RING, ar.AR_ALGO_DIRECT)
        # sizes between buckets use the next bucket up
        if k > 12:
            assert ar.ar_tune((1 << (k - 1)) + 1, dtype=dtype) == d
        prev = d
    # beyond the table: the last / first rows
    assert ar.ar_tune(1 << 30, dtype=dtype) == ar.ar_tune(1 << 27, dtype=dtype)
    assert ar.ar_tune(1, dtype=dtype) == ar.ar_tune(1 << 12, dtype=dtype)
    assert prev is not None


def test_bf16_plans_consult_the_bf16_rows():
    # a bf16 plan asks with msg_bytes = count * 2 and dtype bf16; the
    # geometry it resolves is the bf16 row's
    count = (32 << 20) // 2
    want = ar.ar_tune(32 << 20, dtype="bf16")
    g = ar.ar_plan_geometry(ar.make_desc(8, count, "bf16", "auto", 0, algo="ring"))
    assert (g["proto"], g["nchannels"], g["nwaves"]) == (want["proto"], want["nchannels"], want["nwaves"])


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
@pytest.mark.parametrize("coll", (ar.AR_COLL_REDUCESCATTER, ar.AR_COLL_ALLGATHER))
def test_builtin_table_per_collective(coll, dtype):
    # ReduceScatter and AllGather have tables of their own (one per data
    # type), keyed on the bytes of one rank's full buffer, with the same
    # bucket rule as AllReduce.
    for k in range(12, 28):
        d = ar.ar_tune(1 << k, coll=coll, dtype=dtype)
        assert d["algo"] in (ar.AR_ALGO_RING, ar.AR_ALGO_DIRECT)
        assert 1 <= d["nchannels"] <= ar.AR_MAX_CHANNELS and 1 <= d["nwaves"] <= ar.AR_MAX_WAVES
        if k > 12:
            assert ar.ar_tune((1 << (k - 1)) + 1, coll=coll, dtype=dtype) == d
    assert ar.ar_tune(1 << 30, coll=coll, dtype=dtype) == ar.ar_tune(1 << 27, coll=coll, dtype=dtype)
    # a plan asks with msg_bytes = nranks * count * element size
    n, count = 8, (1 << 20) // 4 // 8
    g = ar.ar_plan_geometry(ar.make_desc(n, count, "f32", "auto", 0, coll=
                                         {ar.AR_COLL_REDUCESCATTER: "reducescatter",
                                          ar.AR_COLL_ALLGATHER: "allgather"}[coll], algo="auto"))
    assert g["algo"] == ar.ar_tune(1 << 20, coll=coll)["algo"]


def test_unknown_collective_defers_to_default():
    assert ar.ar_tune(1 << 20, coll=7) == ar.ar_tune(1 << 20, coll=7)
    ar.ar_set_tuner("fixed_default")
    dflt = ar.ar_tune(1 << 20)
    ar.ar_set_tuner(None)
    assert ar.ar_tune(1 << 20, coll=7) == dflt


def test_fixed_default_and_noop():
    ar.ar_set_tuner("fixed_default")
    d = ar.ar_tune(1 << 20)
    assert (d["proto"], d["nchannels"]) == (ar.AR_PROTO_SIMPLE, 16)
    ar.ar_set_tuner("noop")
    assert ar.ar_tune(1 << 20) == d  # no opinion -> the default
    ar.ar_set_tuner(None)


def test_max_channel_clamp():
    ar.ar_set_tuner(lambda ctx: {"proto": ar.AR_PROTO_LL, "nchannels": 1000})
    d = ar.ar_tune(1 << 20, max_channels=12)
    assert d["proto"] == ar.AR_PROTO_LL and d["nchannels"] == 12
    ar.ar_set_tuner(None)


@pytest.mark.parametrize("bad", [
    {"rc": 1, "proto": ar.AR_PROTO_LL, "nchannels": 4},   # tuner reports failure
    {"proto": 7, "nchannels": 4},                          # protocol out of range
    {"proto": ar.AR_PROTO_LL, "nchannels": -3},            # negative channels
    None,                                                  # callback returns nothing
])
def test_invalid_tuner_output_falls_back(bad):
    ar.ar_set_tuner(lambda ctx: bad)
    d = ar.ar_tune(1 << 22)
    assert (d["proto"], d["nchannels"]) == (ar.AR_PROTO_SIMPLE, 16)
    ar.ar_set_tuner(None)


def test_tuner_sees_context():
    seen = {}

    def t(ctx):
        seen.update(ctx)
        return {"proto": ar.AR_PROTO_LL128, "nchannels": 3, "chunk_bytes": 1000, "nwaves": 99}

    ar.ar_set_tuner(t)
    d = ar.ar_tune(12345, nranks=5, dtype="bf16", max_channels=40, comm_id=77)
    ar.ar_set_tuner(None)
    assert seen == {"coll": 0, "msg_bytes": 12345, "nranks": 5, "dtype": ar.AR_BFLOAT16,
                    "max_channels": 40, "comm_id": 77}
    assert d == {"proto": ar.AR_PROTO_LL128, "proto_name": "ll128", "nchannels": 3,
                 "chunk_bytes": 992, "nwaves": ar.AR_MAX_WAVES, "algo": ar.AR_ALGO_RING, "algo_name": "ring",
                 "direct_parts": 0, "direct_nwaves": 0, "direct_unroll": 0}


def test_tune_rejects_bad_context():
    L = ar.lib()
    out = ar.ar_tune_out()
    assert L.ar_tune(None, ctypes.byref(out)) == ar.AR_ERR_ARG
    ctx = ar.ar_tune_ctx(0, 100, 0, 0, 8, 0)
    assert L.ar_tune(ctypes.byref(ctx), ctypes.byref(out)) == ar.AR_ERR_ARG
    ctx = ar.ar_tune_ctx(0, 100, 8, 5, 8, 0)
    assert L.ar_tune(ctypes.byref(ctx), ctypes.byref(out)) == ar.AR_ERR_ARG


def test_tuner_decision_latency_is_small():
    """Host decision cost (context for the paper's per-decision figures)."""
    L = ar.lib()
    ctx = ar.ar_tune_ctx(0, 1 << 23, 8, 0, 64, 0)
    out = ar.ar_tune_out()
    f = L.ar_tune
    pc, po = ctypes.byref(ctx), ctypes.byref(out)
    t0 = time.perf_counter()
    for _ in range(20000):
        f(pc, po)
    dt = (time.perf_counter() - t0) / 20000
    # dominated by the ctypes call itself; the C decision is tens of ns
    assert dt < 50e-6


# --------------------------------------------------------------- geometry

@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_geometry_segment_rule_matches_oracle(dtype):
    e = 4 if dtype == "f32" else 2
    rng = np.random.default_rng(0)
    counts = [1, 2, 3, 7, 8, 15, 16, 17, 1000, 1023, 1024, 4099, 65537] + list(rng.integers(1, 1 << 24, 20))
    for n in (2, 3, 5, 8, 16):
        for count in counts:
            for proto in ("ll", "ll128", "simple"):
                for nch in (1, 3, 16, 64):
                    g = ar.ar_plan_geometry(ar.make_desc(n, int(count), dtype, proto, nch, 4096))
                    A = 16 // e
                    assert g["seg_elems"] == ro.segment_elems(n, int(count), e)
                    assert g["grid"] == nch * n and g["block"] == 64 * g["nwaves"]
                    assert g["chan_elems"] % A == 0 and g["chan_elems"] * nch >= g["seg_elems"]
                    assert g["chunk_elems"] % A == 0 and g["chunk_elems"] <= g["chan_elems"]
                    assert g["nchunks"] * g["chunk_elems"] >= g["chan_elems"]
                    assert (g["nchunks"] - 1) * g["chunk_elems"] < g["chan_elems"]
                    assert g["wave_elems"] * g["nwaves"] >= g["chunk_elems"]
                    # the peer-direct Simple ring starts each chain with a peer read
                    assert g["msgs_per_run"] == g["nchunks"] * (2 * n - 2 - g["peer_direct"])
                    wire = {"ll": 8 * g["wave_elems"], "simple": 4 * g["wave_elems"],
                            "ll128": -(-4 * g["wave_elems"] // 120) * 128}[proto]
                    assert g["slot_bytes"] >= wire and g["slot_bytes"] % 256 == 0
                    conns = nch * n * g["nwaves"]
                    assert g["fifo_bytes"] == conns * g["fifo_depth"] * g["slot_bytes"]


def test_geometry_trivial_cases():
    g = ar.ar_plan_geometry(ar.make_desc(1, 1000, "f32", "simple", 4))
    assert g["grid"] == 0 and g["fifo_bytes"] == 0
    g = ar.ar_plan_geometry(ar.make_desc(8, 0, "f32", "simple", 4))
    assert g["grid"] == 0


@pytest.mark.parametrize("kw,code", [
    (dict(nranks=0), ar.AR_ERR_ARG),
    (dict(nranks=17), ar.AR_ERR_ARG),
    (dict(dtype=5), ar.AR_ERR_ARG),
    (dict(proto=9), ar.AR_ERR_ARG),
    (dict(nchannels=-1), ar.AR_ERR_ARG),
    (dict(nchannels=300), ar.AR_ERR_ARG),
    (dict(fifo_depth=1), ar.AR_ERR_ARG),
    (dict(nwaves=17), ar.AR_ERR_ARG),
    (dict(placement=3), ar.AR_ERR_ARG),
    (dict(chunk_bytes=1 << 30), ar.AR_ERR_ARG),
    (dict(nchannels=20, max_channels=10), ar.AR_ERR_OCCUPANCY),
    # LL flags are 32-bit: a plan whose slots could hold a line 2^31 messages
    # old is refused (here 2^28 one-unit chunks x 14 messages x depth 4).
    (dict(count=1 << 33, proto="ll", nchannels=1, nwaves=1, chunk_bytes=16), ar.AR_ERR_UNSUPPORTED),
])
def test_geometry_errors(kw, code):
    base = dict(nranks=8, count=1 << 20, dtype="f32", proto="simple", nchannels=4)
    base.update(kw)
    d = ar.make_desc(**base)
    info = ar.ar_plan_info()
    assert ar.lib().ar_plan_geometry(ctypes.byref(d), ctypes.byref(info)) == code


def test_auto_geometry_uses_tuner():
    ar.ar_set_tuner(lambda ctx: {"proto": ar.AR_PROTO_LL, "nchannels": 6, "chunk_bytes": 2048, "nwaves": 2})
    g = ar.ar_plan_geometry(ar.make_desc(8, 1 << 20, "f32", "auto"))
    ar.ar_set_tuner(None)
    assert (g["proto"], g["nchannels"], g["chunk_elems"], g["nwaves"]) == (ar.AR_PROTO_LL, 6, 512, 2)


# ------------------------------------------------------------- bandwidth

def test_bus_bandwidth_matches_paper_pair():
    # The paper quotes ~394 us for a 128 MiB 8-GPU AllReduce (section 5.1)
    # and 596.9 GB/s bus bandwidth for it (section 5.3, Table 2): with
    # busBW = S/t * 2(N-1)/N the two agree.
    t = 128 * 2 ** 20 / (596.9e9 / (2 * 7 / 8))
    assert abs(t * 1e6 - 394) < 1.0
    assert abs(ar.bus_bandwidth(128 * 2 ** 20, 394e-6, 8) - 596.9) < 1.6


def test_ring_byte_counts():
    S = 1 << 20
    assert ar.ring_bytes(S, 8, "f32", "simple") == 44 * S
    assert ar.ring_bytes(S, 8, "f32", "ll") == 72 * S
    assert abs(ar.ring_bytes(S, 8, "f32", "ll128") - (16 + 28 * 128 / 120) * S) < 1
    assert ar.ring_bytes(S, 8, "bf16", "simple") == 58 * S
    assert ar.compulsory_bytes(S, 8) == 16 * S
    # The peer-direct Simple ring: 8 ranks fp32 34 S, bf16 46 S; with 2 ranks
    # the owner reads both inputs and writes both outputs (4 S).
    assert ar.ring_bytes(S, 8, "f32", "simple", peer_direct=True) == 34 * S
    assert ar.ring_bytes(S, 8, "bf16", "simple", peer_direct=True) == 46 * S
    assert ar.ring_bytes(S, 2, "f32", "simple", peer_direct=True) == 4 * S
    # 3 ranks fp32: second rank 12 B, owner 16 B, forwarder 8 B per element
    assert ar.ring_bytes(S, 3, "f32", "simple", peer_direct=True) == 9 * S
    # The peer-direct LL ring only starts its chains with a peer read: the
    # first hop's fp32 partial line (8 B) is neither written nor read.
    assert ar.ring_bytes(S, 8, "f32", "ll", peer_direct=True) == 68 * S
    assert ar.ring_bytes(S, 8, "bf16", "ll", peer_direct=True) == ar.ring_bytes(S, 8, "bf16", "ll") - 8 * S
    # LL128 likewise: its first partial line (8 B per element x 128/120)
    assert abs(ar.ring_bytes(S, 8, "f32", "ll128", peer_direct=True)
               - (ar.ring_bytes(S, 8, "f32", "ll128") - 2 * S * 128 / 120)) < 1


def test_direct_unroll_resolution():
    def geom(count, **kw):
        return ar.ar_plan_geometry(ar.make_desc(8, count, "f32", algo="direct", **kw))
    # by size, when the tuner has no opinion: two units per thread up to
    # 8 MiB per rank, one above
    ar.ar_set_tuner(lambda ctx: {"proto": ar.AR_PROTO_SIMPLE, "nchannels": 4, "algo": ar.AR_ALGO_DIRECT,
                                 "direct_unroll": 0})
    try:
        assert geom((8 << 20) // 4)["direct_unroll"] == 2
        assert geom((8 << 20) // 4 + 4)["direct_unroll"] == 1
    finally:
        ar.ar_set_tuner(None)
    assert geom(1 << 20, direct_unroll=1)["direct_unroll"] == 1
    assert geom(1 << 28, direct_unroll=2)["direct_unroll"] == 2
    # more than 8 ranks: one unit
    g = ar.ar_plan_geometry(ar.make_desc(9, 1 << 10, "f32", algo="direct", direct_unroll=2))
    assert g["direct_unroll"] == 1
    d = ar.make_desc(8, 1 << 10, "f32", algo="direct", direct_unroll=3)
    assert ar.lib().ar_plan_geometry(ctypes.byref(d), ctypes.byref(ar.ar_plan_info())) == ar.AR_ERR_ARG
    # a tuner's choice is used, and an out-of-range one falls back
    ar.ar_set_tuner(lambda ctx: {"proto": ar.AR_PROTO_SIMPLE, "nchannels": 4, "algo": ar.AR_ALGO_DIRECT,
                                 "direct_unroll": 1})
    try:
        assert geom(1 << 10)["direct_unroll"] == 1
        ar.ar_set_tuner(lambda ctx: {"proto": ar.AR_PROTO_SIMPLE, "nchannels": 4, "algo": ar.AR_ALGO_DIRECT,
                                     "direct_unroll": 5})
        assert ar.ar_tune(1 << 10)["algo"] == ar.AR_ALGO_RING  # invalid output -> fixed default
    finally:
        ar.ar_set_tuner(None)


def test_direct_allgather_mode_in_geometry():
    def geom(proto, coll="allreduce", flags=0):
        return ar.ar_plan_geometry(ar.make_desc(8, 1 << 16, "f32", proto, 4, coll=coll, flags=flags, algo="ring"))
    assert geom("simple")["peer_direct"] == 1
    assert geom("simple", "allgather")["peer_direct"] == 1
    assert geom("simple", "reducescatter")["peer_direct"] == 1
    assert geom("simple", flags=ar.AR_PLAN_FIFO_ONLY)["peer_direct"] == 0
    for proto in ("ll", "ll128"):
        assert geom(proto)["peer_direct"] == 1 and geom(proto, flags=ar.AR_PLAN_FIFO_ONLY)["peer_direct"] == 0
        assert geom(proto, "allgather")["peer_direct"] == 1
    # one message fewer per chunk when a chain starts with a peer read
    for proto in ("simple", "ll", "ll128"):
        for coll, per_chunk in (("allreduce", 2 * 8 - 2), ("reducescatter", 8 - 1), ("allgather", 8 - 1)):
            d, f = geom(proto, coll), geom(proto, coll, flags=ar.AR_PLAN_FIFO_ONLY)
            assert f["msgs_per_run"] == f["nchunks"] * per_chunk
            assert d["msgs_per_run"] == d["nchunks"] * (per_chunk - (coll != "allgather"))
    # fp32: the same link bytes either way (the first link carries 4 bytes either way)
    assert geom("simple")["wire_bytes_per_run"] == geom("simple", flags=ar.AR_PLAN_FIFO_ONLY)["wire_bytes_per_run"]
    # LL: the first link carries the chain start's 4 bytes without line flags
    # instead of a 4-byte partial in an 8-byte line (count elements per run)
    assert (geom("ll", flags=ar.AR_PLAN_FIFO_ONLY)["wire_bytes_per_run"] - geom("ll")["wire_bytes_per_run"]
            == (1 << 16) * 4)
    # AllGather has no chain start: the same link bytes either way
    assert geom("ll", "allgather")["wire_bytes_per_run"] == geom("ll", "allgather",
                                                                  flags=ar.AR_PLAN_FIFO_ONLY)["wire_bytes_per_run"]
    d = ar.make_desc(8, 1 << 16, "f32", "simple", 4, flags=8)
    assert ar.lib().ar_plan_geometry(ctypes.byref(d), ctypes.byref(ar.ar_plan_info())) == ar.AR_ERR_ARG
    # the ordered-read flag of LL128 changes no geometry
    assert geom("ll128", flags=ar.AR_PLAN_LL128_ORDERED) == geom("ll128")


def test_default_fifo_depth_deepens_small_runs():
    """Without an explicit depth a run with more messages than slots gets a
    deeper FIFO (up to 16) while the FIFO stays within 4 MiB; large runs keep
    the protocol's depth; an explicit depth is kept as given."""
    def geom(count, proto, nch, depth=0):
        return ar.ar_plan_geometry(ar.make_desc(8, count, "f32", proto, nch, 0, fifo_depth=depth, algo="ring"))
    for proto, base in (("simple", 2), ("ll", 4), ("ll128", 4)):
        small = geom(1024, proto, 1)
        assert small["fifo_depth"] == 16 and small["msgs_per_run"] <= 16
        big = geom(1 << 25, proto, 64)
        assert big["fifo_depth"] == base
        assert geom(1024, proto, 1, depth=3)["fifo_depth"] == 3
        for g in (small, big):
            conns = g["nchannels"] * 8 * g["nwaves"]
            assert g["fifo_bytes"] == conns * g["fifo_depth"] * g["slot_bytes"]
            # deepened only while the doubled FIFO fits the budget
            if g["fifo_depth"] > base:
                assert g["fifo_bytes"] <= 4 << 20
    # a run whose messages already fit keeps the protocol's depth (2 ranks:
    # 2 LL messages, 1 peer-direct Simple message per run)
    for proto, base in (("simple", 2), ("ll", 4)):
        g = ar.ar_plan_geometry(ar.make_desc(2, 1024, "f32", proto, 1, 0, algo="ring"))
        assert g["msgs_per_run"] <= base and g["fifo_depth"] == base


# ------------------------------------------------------------- algorithms

def test_direct_geometry_and_algorithm_choice():
    g = ar.ar_plan_geometry(ar.make_desc(8, 1 << 20, "f32", algo="direct"))
    assert g["algo"] == ar.AR_ALGO_DIRECT and g["fifo_bytes"] == 0 and g["msgs_per_run"] == 0
    assert g["grid"] == 8 * g["nchannels"] and g["seg_elems"] == ro.segment_elems(8, 1 << 20, 4)
    assert g["chan_elems"] * g["nchannels"] >= g["seg_elems"]
    # a requested protocol implies the ring; direct with a protocol is an error
    g = ar.ar_plan_geometry(ar.make_desc(8, 1 << 20, "f32", "ll", 4))
    assert g["algo"] == ar.AR_ALGO_RING
    info = ar.ar_plan_info()
    d = ar.make_desc(8, 1 << 20, "f32", "simple", 4, algo="direct")
    assert ar.lib().ar_plan_geometry(ctypes.byref(d), ctypes.byref(info)) == ar.AR_ERR_ARG
    d = ar.make_desc(8, 1 << 20, "f32", algo=7)
    assert ar.lib().ar_plan_geometry(ctypes.byref(d), ctypes.byref(info)) == ar.AR_ERR_ARG
    # the tuner's algorithm choice is honoured under AUTO
    ar.ar_set_tuner(lambda ctx: {"algo": ar.AR_ALGO_DIRECT, "proto": ar.AR_PROTO_SIMPLE, "nchannels": 5})
    assert ar.ar_plan_geometry(ar.make_desc(8, 4096, "f32"))["algo"] == ar.AR_ALGO_DIRECT
    # ... while the ring columns of that answer still serve a forced ring
    g = ar.ar_plan_geometry(ar.make_desc(8, 4096, "f32", algo="ring"))
    assert g["algo"] == ar.AR_ALGO_RING and g["nchannels"] == 5
    ar.ar_set_tuner(lambda ctx: {"algo": 9, "proto": ar.AR_PROTO_LL, "nchannels": 5})
    assert ar.ar_tune(4096)["algo"] == ar.AR_ALGO_RING and ar.ar_tune(4096)["nchannels"] == 16
    ar.ar_set_tuner(None)


def test_table_rows_scale_with_rank_count():
    """Rows measured with 8 ranks keep their workgroup count at other rank
    counts: channels and direct parts scale by 8/N (at least 1, 0 stays the
    library's rule); with two ranks LL rows defer to the default."""
    for size in (4096, 1 << 20, 4 << 20, 128 << 20):
        base = ar.ar_tuner_raw("table", size, nranks=8)
        for n in (2, 3, 4, 5, 16):
            t = ar.ar_tuner_raw("table", size, nranks=n)
            assert t["rc"] == 0 and t["algo"] == base["algo"]
            assert t["direct_nwaves"] == base["direct_nwaves"] and t["direct_unroll"] == base["direct_unroll"]
            want_parts = max(1, (base["direct_parts"] * 8 + n // 2) // n) if base["direct_parts"] else 0
            assert t["direct_parts"] == want_parts, (size, n, t, base)
            if n == 2 and base["proto"] == ar.AR_PROTO_LL:
                assert t["proto"] == ar.AR_PROTO_AUTO and t["nchannels"] == 0
            else:
                assert t["proto"] == base["proto"] and t["chunk_bytes"] == base["chunk_bytes"]
                assert t["nchannels"] == max(1, (base["nchannels"] * 8 + n // 2) // n), (size, n, t, base)
    # 8 ranks: the rows as tabulated
    assert ar.ar_tuner_raw("table", 128 << 20, nranks=8)["nchannels"] == 64
