"""GPU parity: the HIP simulated-ring AllReduce against the CPU oracle.

Every case runs through the C ABI (ar_plan_ex / ar_run via the ctypes
binding) and compares every rank's output with the oracle element by
element: bit-exact for fp32 and for bf16 (fp32 accumulation, one rounding).
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from oracle import ring_oracle as ro
from tests.gpu_helpers import assert_ranks_equal, draw, oracle_bits, run_case, say, to_bits, to_device

pytestmark = pytest.mark.gpu

PROTOS = ("simple", "ll", "ll128")


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


# ------------------------------------------- D1: 4 KiB fp32, integer values, one channel

def test_d1_simple_one_channel_bitexact(ar):
    w = workloads.WORKLOADS["D1"]
    x = w.draw()
    info = run_case(ar, x, "f32", "D1", proto="simple", nchannels=1, chunk_bytes=1024)
    assert info["proto"] == ar.AR_PROTO_SIMPLE and info["nchannels"] == 1
    # integer-valued inputs: the result is the exact integer sum
    import torch  # noqa: F401

    y = ro.allreduce_f32(x)
    assert np.array_equal(y.astype(np.int64), x.astype(np.int64).sum(axis=0))


# --------------------------------------------------------- small-size grid

SMALL_COUNTS = (1, 5, 64, 1000, 4099, 65537)


@pytest.mark.parametrize("proto", PROTOS)
@pytest.mark.parametrize("dtype", ("f32", "bf16"))
@pytest.mark.parametrize("n", (2, 3, 8))
def test_small_grid(ar, proto, dtype, n):
    for count in SMALL_COUNTS:
        x = draw(n, count, dtype, "normal", seed=1000 + n * 31 + count)
        for nch in (1, 3):
            run_case(ar, x, dtype, f"grid-{proto}-{dtype}-{n}-{count}-{nch}", proto=proto, nchannels=nch)


def test_ll128_line_tails(ar):
    """LL128 messages that end at every position of a 128-byte line, in
    both line formats (30 fp32 values or partials per line, 60 bf16
    values): inside lane 6's part, inside lane 7's half-width part (which
    moves on an access that starts inside lane 6's), and at every other
    lane.  One channel and one wave, so a message is a whole segment and
    the last segment's length walks through every remainder.  Segments of
    about 240 elements (8 to 17 reduce-scatter lines) run the two-access
    batches; about 1200 elements (40 lines), the four-access ones.  Two
    ranks run both ways: peer-direct (the owner reads the chain start's
    input and sends all-gather lines) and through the FIFOs (a
    reduce-scatter line hop)."""
    for dtype in ("f32", "bf16"):
        for n, step, hi, base in ((2, 1, 124, 240), (3, 3, 190, 240), (2, 1, 124, 1200), (3, 5, 190, 1200)):
            for flags in ((0, ar.AR_PLAN_FIFO_ONLY) if n == 2 else (0,)):
                for r in range(0, hi, step):
                    count = n * base + r
                    x = draw(n, count, dtype, "normal", seed=5000 + 7 * n + r)
                    run_case(ar, x, dtype, f"ll128-tail-{dtype}-{n}-{count}-{flags}", proto="ll128", nchannels=1,
                             nwaves=1, flags=flags)


def test_ll128_ordered_reads(ar):
    """AR_PLAN_LL128_ORDERED: every batch is read after its flags were seen
    current.  Same bits as the oracle for both dtypes, several rank counts,
    ragged counts, one and three channels, and both batch widths (one wave
    per rank, so segments of 60+ elements run four-access batches)."""
    for dtype in ("f32", "bf16"):
        for n in (2, 3, 8):
            for count in (1, 257, 4099, 65537):
                x = draw(n, count, dtype, "normal", seed=3100 + 7 * n + count)
                for nch, nw in ((1, 1), (3, 4)):
                    run_case(ar, x, dtype, f"ll128-ordered-{dtype}-{n}-{count}-{nch}-{nw}", proto="ll128",
                             nchannels=nch, nwaves=nw, flags=ar.AR_PLAN_LL128_ORDERED)


def test_bound_calls(ar):
    """Plan.bind checks the buffers once and returns a single-C-call
    launcher: repeated calls out of place and a call in place give the
    oracle's bits, and a call after the plan is destroyed raises."""
    import torch

    n, count = 8, 40000
    x = draw(n, count, "f32", "uniform", seed=4242)
    want = oracle_bits(x, "f32")
    for algo in ("ring", "direct"):
        say(f"bound calls, {algo}")
        plan = ar.Plan(n, count, "f32", algo=algo)
        send = to_device(x, "f32")
        recv = [torch.empty_like(t) for t in send]
        fn = plan.bind(send, recv)
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        assert_ranks_equal(recv, want, "f32", f"bound out of place, {algo}")
        ts = to_device(x, "f32")
        plan.bind(ts)()
        torch.cuda.synchronize()
        assert_ranks_equal(ts, want, "f32", f"bound in place, {algo}")
        with pytest.raises(ValueError):
            plan.bind(send[:-1], recv)
        plan.destroy()
        with pytest.raises(ar.ARError):
            fn()


@pytest.mark.parametrize("n", (1, 4, 5, 16))
def test_rank_counts(ar, n):
    for proto in PROTOS:
        for dtype in ("f32", "bf16"):
            x = draw(n, 12345, dtype, "uniform", seed=77 + n)
            run_case(ar, x, dtype, f"ranks-{n}-{proto}-{dtype}", proto=proto, nchannels=2)


def test_all_ones_gives_n(ar):
    import torch

    for proto in PROTOS:
        for n in (2, 7, 8):
            x = workloads.draw(n, 50000, "f32", "ones", 0)
            ts = to_device(x, "f32")
            plan = ar.Plan(n, 50000, "f32", proto=proto, nchannels=4)
            plan.run(ts)
            torch.cuda.synchronize()
            for t in ts:
                assert bool((t == float(n)).all())
            plan.destroy()


ORDER_VALUES = np.array([2.0 ** 24, -(2.0 ** 24), 2.0 ** 25, 1.0, -1.0, 3.0, 0.5], np.float32)


def order_input(n, count, dtype, seed):
    """Order-revealing inputs: large values that cancel and small ones that
    a large partial absorbs, so different chain orders give different sums.
    Every value is exact in bf16, so the bf16 case carries the same values."""
    import torch

    rng = np.random.default_rng(seed)
    xf = rng.choice(ORDER_VALUES, size=(n, count)).astype(np.float32)
    if dtype == "f32":
        return xf
    xb = torch.from_numpy(xf).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ro.bf16_to_f32(xb), xf)
    return xb


def test_order_revealing_brute_force(ar):
    """Tiny inputs whose chain orders all differ: each element must equal the
    chain that starts at its segment's rank."""
    rng = np.random.default_rng(5)
    for n in (2, 3, 4, 8):
        for count in (4, 13, 64, 257):
            x = rng.choice(ORDER_VALUES, size=(n, count)).astype(np.float32)
            for proto in PROTOS:
                run_case(ar, x, "f32", f"order-{n}-{count}-{proto}", proto=proto, nchannels=2, chunk_bytes=64)


def test_order_revealing_bf16(ar):
    """bf16 with fp32 accumulation on order-revealing inputs: the chain of
    every 8-element-aligned segment must start at its own rank and run in
    ring order, on the ring under each protocol (each both peer-direct and
    FIFO only) and on the direct algorithm.  The inputs
    are checked to be informative: starting every chain one rank earlier
    changes many rounded results."""
    informative = 0
    cfgs = [dict(proto=p, nchannels=2, chunk_bytes=64) for p in PROTOS]
    cfgs += [dict(proto=p, nchannels=3, chunk_bytes=32, flags=2) for p in PROTOS]
    cfgs += [dict(algo="direct"), dict(algo="direct", nchannels=3, nwaves=1)]
    for n in (2, 3, 4, 8):
        for count in (16, 40, 64, 264, 1001):
            x = order_input(n, count, "bf16", seed=900 + 17 * n + count)
            informative += int(np.count_nonzero(ro.allreduce_bf16(x) != ro.allreduce_bf16(np.roll(x, 1, axis=0))))
            for cfg in cfgs:
                run_case(ar, x, "bf16", f"order-bf16-{n}-{count}-{cfg}", **cfg)
    assert informative > 200, informative


def test_order_revealing_bf16_full_size(ar):
    """The bf16 chain order at the 32 MiB bf16 workload's size (8 ranks x
    16 Mi elements): order-revealing values, compared on the device under
    the table's ring and overall choices, the fixed default, LL and LL128."""
    import torch

    n, count = 8, 16 << 20
    x = order_input(n, count, "bf16", seed=4711)
    want = ro.allreduce_bf16(x)
    changed = int(np.count_nonzero(want != ro.allreduce_bf16(np.roll(x, 1, axis=0))))
    assert changed > count // 20, changed  # about 8.6 % of the elements
    want_dev = to_device(want[None, :], "bf16")[0]
    base = to_device(x, "bf16")
    del x
    for cfg in (dict(proto="auto", algo="ring"), dict(proto="auto"), dict(proto="simple", nchannels=16),
                dict(proto="ll", nchannels=64), dict(proto="ll128", nchannels=64)):
        say(f"order bf16 full size {cfg}")
        out = [torch.empty_like(t) for t in base]
        plan = ar.Plan(n, count, "bf16", **cfg)
        plan.run_oop(base, out)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK, cfg
        plan.destroy()
        for r in range(n):
            if not torch.equal(out[r].view(torch.int16), want_dev.view(torch.int16)):
                bad = (out[r].view(torch.int16) != want_dev.view(torch.int16)).nonzero()
                raise AssertionError(f"{cfg} rank {r}: {bad.numel()} elements differ, first {int(bad[0])}")


# ------------------------------------------------- layout independence (U1)

def _metamorphic_configs():
    cfgs = []
    for proto in PROTOS:
        for nch in (1, 2, 5, 16, 64):
            for chunk in (16, 4096, 1 << 20):
                cfgs.append(dict(proto=proto, nchannels=nch, chunk_bytes=chunk))
    cfgs += [dict(proto="simple", nchannels=8, nwaves=w) for w in (1, 2, 8, 16)]
    cfgs += [dict(proto=p, nchannels=16, placement=1) for p in PROTOS]
    cfgs += [dict(proto=p, nchannels=4, fifo_depth=d) for p in PROTOS for d in (2, 3, 8)]
    # every hop through the FIFOs instead of the peer-direct mode: the Simple
    # ring's all-gather and every protocol's chain starts
    cfgs += [dict(proto=p, nchannels=nch, chunk_bytes=chunk, flags=2) for p in PROTOS
             for nch in (1, 5, 64) for chunk in (16, 4096)]
    cfgs += [dict(proto="auto")]
    return cfgs


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_metamorphic_layouts_identical_bits(ar, dtype):
    import torch

    n, count = 8, 300007
    x = draw(n, count, dtype, "normal", seed=4242)
    want = oracle_bits(x, dtype)
    base = to_device(x, dtype)
    for cfg in _metamorphic_configs():
        say(f"metamorphic {dtype} {cfg}")
        ts = [t.clone() for t in base]
        plan = ar.Plan(n, count, dtype, **cfg)
        plan.run(ts)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        assert_ranks_equal(ts, want, dtype, str(cfg))
        plan.destroy()


# ------------------------------------------------ full-size configurations

def _device_compare(ts, want_dev, dtype):
    import torch

    iv = torch.int32 if dtype == "f32" else torch.int16
    for r, t in enumerate(ts):
        if not torch.equal(t.view(iv), want_dev.view(iv)):
            bad = (t.view(iv) != want_dev.view(iv)).nonzero()
            raise AssertionError(f"rank {r}: {bad.numel()} elements differ, first {int(bad[0])}")


def _full_size_sweep(ar, wl, cfgs):
    import torch

    x = wl.draw()
    dtype = wl.dtype
    want = oracle_bits(x, dtype)
    want_dev = to_device(want[None, :].view(np.float32 if dtype == "f32" else np.uint16), dtype)[0]
    base = to_device(x, dtype)
    del x
    for cfg in cfgs:
        say(f"{wl.name} {cfg}")
        ts = [t.clone() for t in base]
        plan = ar.Plan(wl.nranks, wl.count, dtype, **cfg)
        plan.run(ts)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK, cfg
        _device_compare(ts, want_dev, dtype)
        plan.destroy()
        del ts


def test_d2_ll_vs_simple_channels(ar):
    wl = workloads.WORKLOADS["D2"]
    _full_size_sweep(ar, wl, [dict(proto=p, nchannels=c) for p in ("ll", "simple") for c in wl.channels])


def test_d3_bf16_simple_chunks_channels(ar):
    wl = workloads.WORKLOADS["D3"]
    cfgs = [dict(proto="simple", nchannels=c, chunk_bytes=k) for c in wl.channels for k in wl.chunks]
    # and the built-in bf16 table's own choices, ring and overall
    cfgs += [dict(proto="auto", algo="ring"), dict(proto="auto", algo="auto")]
    _full_size_sweep(ar, wl, cfgs)


def test_d5_ll128_vs_simple(ar):
    wl = workloads.WORKLOADS["D5"]
    _full_size_sweep(ar, wl, [dict(proto=p, nchannels=c) for p in ("ll128", "simple") for c in wl.channels])


def test_d4_size_sweep_tuned_and_default(ar):
    import torch

    for size in workloads.WORKLOADS["D4"].extra["sizes"]:
        wl = workloads.sweep_workload(size)
        x = wl.draw()
        want = oracle_bits(x, "f32")
        want_dev = torch.from_numpy(want.view(np.float32)).to("cuda:0")
        base = to_device(x, "f32")
        # the table's overall choice, its ring choice (protocol, channels,
        # chunk, waves for this size) and the fixed default
        for cfg in (dict(proto="auto"), dict(proto="auto", algo="ring"), dict(proto="simple", nchannels=16)):
            say(f"D4 {size} {cfg}")
            ts = [t.clone() for t in base]
            plan = ar.Plan(8, wl.count, "f32", **cfg)
            plan.run(ts)
            torch.cuda.synchronize()
            assert plan.status() == ar.AR_OK
            _device_compare(ts, want_dev, "f32")
            plan.destroy()


def test_fp64_normwise_bound_full_size(ar):
    import torch

    wl = workloads.WORKLOADS["D2"]
    x = wl.draw()
    ts = to_device(x, "f32")
    plan = ar.Plan(8, wl.count, "f32", proto="auto")
    plan.run(ts)
    torch.cuda.synchronize()
    y = ts[3].cpu().numpy().astype(np.float64)
    err = np.abs(y - ro.sum_f64(x))
    scale = ro.abs_sum_f64(x)
    assert np.all(err <= ro.recursive_sum_gamma(8) * scale)
    assert np.all(err <= 1e-5 * scale)
    plan.destroy()


# ------------------------------------------------ in place, repeats, epochs

@pytest.mark.parametrize("proto", PROTOS)
def test_out_of_place_equals_in_place(ar, proto):
    import torch

    n, count, dtype = 8, 100003, "f32"
    x = draw(n, count, dtype, "normal", seed=9)
    want = oracle_bits(x, dtype)
    send = to_device(x, dtype)
    recv = [torch.full_like(t, float("nan")) for t in send]
    plan = ar.Plan(n, count, dtype, proto=proto, nchannels=4)
    plan.run_oop(send, recv)
    torch.cuda.synchronize()
    assert_ranks_equal(recv, want, dtype, "oop")
    # inputs untouched
    for r in range(n):
        assert np.array_equal(to_bits(send[r], dtype), x[r].view(np.uint32))
    plan.destroy()


@pytest.mark.parametrize("proto", PROTOS)
@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_repeated_runs_poisoned_fifo(ar, proto, dtype):
    """Back-to-back runs of one plan with the FIFO poisoned (0xFF) before each
    run: a reader that consumed a slot before its writer filled it would see
    NaN.  Flag epochs advance across runs with no reset."""
    import torch

    n, count = 8, 40000
    plan = ar.Plan(n, count, dtype, proto=proto, nchannels=3, fifo_depth=2)
    for it in range(30):
        x = draw(n, count, dtype, "normal", seed=500 + it)
        ts = to_device(x, dtype)
        plan.poison()
        plan.run(ts)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        assert_ranks_equal(ts, oracle_bits(x, dtype), dtype, f"repeat {it}")
    plan.destroy()


@pytest.mark.parametrize("proto", PROTOS)
def test_jitter_keeps_results(ar, proto):
    for seed in range(3):
        x = draw(8, 70001, "f32", "normal", seed=600 + seed)
        run_case(ar, x, "f32", f"jitter-{proto}", poison=True, proto=proto, nchannels=4,
                 debug_flags=ar.AR_DEBUG_JITTER)


def test_many_runs_one_stream(ar):
    """Many runs queued on one stream without synchronising in between."""
    import torch

    n, count = 8, 65536
    x = draw(n, count, "f32", "normal", seed=77)
    base = to_device(x, "f32")
    want = oracle_bits(x, "f32")
    for proto in PROTOS:
        plan = ar.Plan(n, count, "f32", proto=proto, nchannels=8)
        outs = []
        for _ in range(200):
            ts = [t.clone() for t in base]
            plan.run(ts)
            outs.append(ts)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        for ts in outs[::37]:
            assert_ranks_equal(ts, want, "f32", f"many-{proto}")
        plan.destroy()


# --------------------------------------------------------- failure handling

@pytest.mark.parametrize("proto", PROTOS)
def test_watchdog_timeout_then_reset(ar, proto):
    """A debug knob suppresses one message announcement; the waiting waves hit
    the (short) watchdog, every wave exits, and the plan reports a timeout
    until it is reset."""
    import torch

    n, count = 8, 20000
    x = draw(n, count, "f32", "normal", seed=1)
    ts = to_device(x, "f32")
    plan = ar.Plan(n, count, "f32", proto=proto, nchannels=2, timeout_us=20000,
                   debug_flags=ar.AR_DEBUG_SKIP_POST)
    plan.run(ts)
    torch.cuda.synchronize()
    assert plan.status() == ar.AR_ERR_TIMEOUT
    with pytest.raises(ar.ARError) as ei:
        plan.run(ts)
    assert ei.value.code == ar.AR_ERR_STATE
    plan.destroy()
    # a normal plan on the same device still works
    run_case(ar, x, "f32", "after-timeout", proto=proto, nchannels=2)


def test_argument_errors(ar):
    import torch

    n, count = 4, 1000
    plan = ar.Plan(n, count, "f32", proto="simple", nchannels=1)
    big = torch.zeros(n * count + 8, device="cuda:0")
    # misaligned buffer
    mis = [big[1 + r * count: 1 + (r + 1) * count] for r in range(n)]
    import ctypes

    arr = (ctypes.c_void_p * n)(*[t.data_ptr() for t in mis])
    assert ar.lib().ar_run(plan.handle, arr, None) == ar.AR_ERR_ARG
    # overlapping buffers
    ov = [big[0:count]] * n
    arr = (ctypes.c_void_p * n)(*[t.data_ptr() for t in ov])
    assert ar.lib().ar_run(plan.handle, arr, None) == ar.AR_ERR_ARG
    # NULL pointer array
    assert ar.lib().ar_run(plan.handle, None, None) == ar.AR_ERR_ARG
    plan.destroy()
    # too many channels for co-residency
    h = ar.lib().ar_plan_ex(ctypes.byref(ar.make_desc(16, 1 << 20, "f32", "simple", 256, nwaves=16)))
    assert not h and ar.ar_last_error() == ar.AR_ERR_OCCUPANCY


# ----------------------------------------------------- device bf16 rounding

def test_device_bf16_rounding_matches_oracle(ar):
    import torch

    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x1234, 0xC000], np.uint32)
    u = ((np.arange(1 << 16, dtype=np.uint32)[:, None] << np.uint32(16)) | lows[None, :]).ravel()
    f = u.view(np.float32)
    got = ar.ar_debug_bf16_round(torch.from_numpy(f.copy()).to("cuda:0"))
    torch.cuda.synchronize()
    got = got.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, ro.f32_to_bf16_rne(f))


# ------------------------------------------- profiler -> tuner closed loop

def test_plan_profiler_hook_records_kernel_time(ar):
    import torch

    ar.ar_profile_clear()
    n, count = 8, 1 << 20
    x = draw(n, count, "f32", "uniform", seed=3)
    ts = to_device(x, "f32")
    plan = ar.Plan(n, count, "f32", proto="simple", nchannels=8, comm_id=777, flags=ar.AR_PLAN_PROFILE)
    assert ar.ar_profile_lookup(777) is None
    plan.run(ts)
    torch.cuda.synchronize()
    assert plan.status() == ar.AR_OK          # harvests the finished run
    st = ar.ar_profile_lookup(777)
    assert st is not None and st["nchannels"] == 8 and 1_000 < st["latency_ns"] < 100_000_000
    assert_ranks_equal(ts, oracle_bits(x, "f32"), "f32", "profiled run")
    plan.destroy()


def test_closed_loop_adaptive_channels_on_gpu(ar):
    """Per-call decisions from the adaptive tuner, fed by the plans' own
    profiler hook: the channel count ramps from 2 to 12 and every result
    stays bit-exact."""
    import torch

    ar.ar_profile_clear()
    ar.ar_set_tuner("adaptive", adaptive={"ramp_calls": 3})
    n, count, comm = 8, 1 << 20, 4242
    x = draw(n, count, "f32", "uniform", seed=11)
    want = oracle_bits(x, "f32")
    base = to_device(x, "f32")
    plans, seen = {}, []
    try:
        for _ in range(45):
            d = ar.ar_tune(count * 4, n, "f32", comm_id=comm)
            key = (d["proto"], d["nchannels"])
            if key not in plans:
                plans[key] = ar.Plan(n, count, "f32", proto=d["proto_name"], nchannels=d["nchannels"],
                                     comm_id=comm, flags=ar.AR_PLAN_PROFILE)
            p = plans[key]
            ts = [t.clone() for t in base]
            p.run(ts)
            torch.cuda.synchronize()
            assert p.status() == ar.AR_OK
            assert_ranks_equal(ts, want, "f32", f"closed loop C={d['nchannels']}")
            seen.append(d["nchannels"])
    finally:
        ar.ar_set_tuner(None)
        for p in plans.values():
            p.destroy()
    assert seen[0] == 2 and seen[-1] == 12, seen


# -------------------------------------------------------- direct algorithm
#
# The direct algorithm sums each segment in the ring's chain order, so its
# results must equal the oracle (and the ring) bit for bit.

@pytest.mark.parametrize("dtype", ("f32", "bf16"))
@pytest.mark.parametrize("n", (2, 3, 8, 9, 16))
def test_direct_small_grid(ar, dtype, n):
    for count in SMALL_COUNTS:
        x = draw(n, count, dtype, "normal", seed=2000 + n * 31 + count)
        for parts in (0, 1, 3):
            for unroll in (1, 2):
                run_case(ar, x, dtype, f"direct-{dtype}-{n}-{count}-{parts}-u{unroll}", algo="direct",
                         nchannels=parts, direct_unroll=unroll)


def test_direct_order_revealing(ar):
    vals = np.array([2.0 ** 24, -(2.0 ** 24), 2.0 ** 25, 1.0, -1.0, 3.0, 0.5], np.float32)
    rng = np.random.default_rng(6)
    for n in (2, 3, 4, 8, 16):
        for count in (4, 13, 64, 257, 5000):
            x = rng.choice(vals, size=(n, count)).astype(np.float32)
            run_case(ar, x, "f32", f"direct-order-{n}-{count}", algo="direct")


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_direct_equals_ring_bits(ar, dtype):
    import torch

    n, count = 8, 300007
    x = draw(n, count, dtype, "normal", seed=4243)
    want = oracle_bits(x, dtype)
    base = to_device(x, dtype)
    for cfg in (dict(algo="direct"), dict(algo="direct", nchannels=1, nwaves=1),
                dict(algo="direct", nchannels=200, nwaves=16), dict(proto="simple", nchannels=7),
                dict(algo="direct", direct_unroll=1), dict(algo="direct", direct_unroll=2, nchannels=5)):
        ts = [t.clone() for t in base]
        plan = ar.Plan(n, count, dtype, **cfg)
        plan.run(ts)
        torch.cuda.synchronize()
        assert_ranks_equal(ts, want, dtype, str(cfg))
        plan.destroy()


def test_direct_full_size(ar):
    _full_size_sweep(ar, workloads.WORKLOADS["D5"], [dict(algo="direct"), dict(algo="direct", nchannels=64)])
    _full_size_sweep(ar, workloads.WORKLOADS["D3"], [dict(algo="direct")])


def test_direct_out_of_place_and_repeats(ar):
    import torch

    n, count = 8, 100003
    x = draw(n, count, "f32", "normal", seed=12)
    want = oracle_bits(x, "f32")
    send = to_device(x, "f32")
    plan = ar.Plan(n, count, "f32", algo="direct")
    for _ in range(3):
        recv = [torch.full_like(t, float("nan")) for t in send]
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        assert_ranks_equal(recv, want, "f32", "direct oop")
    for r in range(n):
        assert np.array_equal(to_bits(send[r], "f32"), x[r].view(np.uint32))
    plan.destroy()


def test_empty_runs_are_no_ops(ar):
    """count = 0: every algorithm and collective accepts empty buffers,
    launches nothing and leaves the plan's status clean; a real run
    afterwards is unaffected."""
    import torch

    for n in (2, 8):
        for cfg in (dict(proto="simple", nchannels=2), dict(proto="ll", nchannels=2),
                    dict(proto="ll128", nchannels=2), dict(algo="direct")):
            for coll in ("allreduce", "reducescatter", "allgather"):
                label = f"empty N={n} {coll} {cfg}"
                say(label)
                plan = ar.Plan(n, 0, "f32", coll=coll, **cfg)
                assert plan.info["grid"] == 0, label
                bufs = [torch.empty(0, device="cuda:0") for _ in range(n)]
                plan.run(bufs)
                plan.run_oop(bufs, [torch.empty(0, device="cuda:0") for _ in range(n)])
                torch.cuda.synchronize()
                assert plan.status() == ar.AR_OK, label
                plan.destroy()
    x = draw(8, 4099, "f32", "normal", seed=3)
    run_case(ar, x, "f32", "after empty runs", proto="simple", nchannels=2)
