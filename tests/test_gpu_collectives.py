"""GPU parity of ReduceScatter and AllGather (ring under each protocol, and
the direct algorithm) against the CPU oracle, bit for bit, out of place and
in the in-place layouts."""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from oracle import ring_oracle as ro
from tests.gpu_helpers import draw, say, to_bits, to_device

pytestmark = pytest.mark.gpu

CFGS = [dict(proto="simple", nchannels=1), dict(proto="simple", nchannels=3, chunk_bytes=256),
        dict(proto="ll", nchannels=2), dict(proto="ll128", nchannels=2),
        dict(algo="direct"), dict(algo="direct", nchannels=3, nwaves=1)]


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


def _bits(ts, dtype):
    return np.stack([to_bits(t, dtype) for t in ts])


def _rs_case(ar, n, count, dtype, cfg, in_place, seed, x=None):
    import torch

    if x is None:
        x = draw(n, n * count, dtype, "normal", seed)
    want = ro.reduce_scatter(x, dtype)
    want = want.view(np.uint32) if dtype == "f32" else want
    plan = ar.Plan(n, count, dtype, coll="reducescatter", **cfg)
    label = f"RS N={n} count={count} {dtype} {cfg} in_place={in_place}"
    say(label)
    if in_place:
        bufs = to_device(x, dtype)
        plan.run(bufs)
        torch.cuda.synchronize()
        got = np.stack([to_bits(bufs[r], dtype)[r * count:(r + 1) * count] for r in range(n)])
    else:
        send = to_device(x, dtype)
        recv = [torch.zeros(count, dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        got = _bits(recv, dtype)
        assert np.array_equal(_bits(send, dtype), x.view(np.uint32) if dtype == "f32" else x), "input changed"
    assert plan.status() == ar.AR_OK
    plan.destroy()
    assert np.array_equal(got, want), label


def _ag_case(ar, n, count, dtype, cfg, in_place, seed):
    import torch

    x = draw(n, count, dtype, "normal", seed)
    want = ro.all_gather(x)
    want = want.view(np.uint32) if dtype == "f32" else want
    plan = ar.Plan(n, count, dtype, coll="allgather", **cfg)
    label = f"AG N={n} count={count} {dtype} {cfg} in_place={in_place}"
    say(label)
    if in_place:
        full = np.zeros((n, n * count), dtype=x.dtype)
        for r in range(n):
            full[r, r * count:(r + 1) * count] = x[r]
        bufs = to_device(full, dtype)
        plan.run(bufs)
        torch.cuda.synchronize()
        got = _bits(bufs, dtype)
    else:
        send = to_device(x, dtype)
        recv = [torch.zeros(n * count, dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        got = _bits(recv, dtype)
    assert plan.status() == ar.AR_OK
    plan.destroy()
    for r in range(n):
        assert np.array_equal(got[r], want), f"{label}: rank {r}"


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
@pytest.mark.parametrize("n", (2, 3, 8, 16))
def test_reduce_scatter(ar, dtype, n):
    a = 4 if dtype == "f32" else 8
    for count in (a, 3 * a, 1000 * a // 8 * 8, 8192):
        for i, cfg in enumerate(CFGS):
            _rs_case(ar, n, count, dtype, cfg, in_place=bool(i % 2), seed=100 * n + count + i)


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_reduce_scatter_order_revealing(ar, dtype):
    """Order-revealing inputs (large values that cancel, small ones a large
    partial absorbs; all exact in bf16): block r must be summed along the
    chain that starts at rank r+1, on the ring under each protocol and on
    the direct algorithm.  Starting the chains one rank earlier would change
    many results, which the test checks first."""
    from tests.test_gpu_parity import order_input

    a = 4 if dtype == "f32" else 8
    informative = 0
    for n in (2, 3, 4, 8):
        for count in (a, 3 * a, 64, 200):
            x = order_input(n, n * count, dtype, seed=700 + 13 * n + count)
            want = ro.reduce_scatter(x, dtype)
            informative += int(np.count_nonzero(want != ro.reduce_scatter(np.roll(x, 1, axis=0), dtype)))
            for i, cfg in enumerate(CFGS):
                _rs_case(ar, n, count, dtype, cfg, in_place=bool(i % 2), seed=0, x=x)
    assert informative > 200, informative


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
@pytest.mark.parametrize("n", (2, 3, 8, 16))
def test_all_gather(ar, dtype, n):
    a = 4 if dtype == "f32" else 8
    for count in (a, 3 * a, 1000 * a // 8 * 8, 8192):
        for i, cfg in enumerate(CFGS):
            _ag_case(ar, n, count, dtype, cfg, in_place=bool(i % 2), seed=200 * n + count + i)


def test_all_gather_keeps_nan_payloads(ar):
    """AllGather is a copy: every bit pattern, NaN payloads included, survives."""
    for cfg in (dict(proto="simple"), dict(proto="ll"), dict(proto="ll128"), dict(algo="direct")):
        for dtype in ("f32", "bf16"):
            n, count = 4, 64
            rng = np.random.default_rng(3)
            if dtype == "f32":
                x = rng.integers(0x7F800001, 0x7FFFFFFF, size=(n, count), dtype=np.uint32).view(np.float32)
            else:
                x = rng.integers(0x7F81, 0x7FFF, size=(n, count), dtype=np.uint16)
            import torch

            send = to_device(x, dtype)
            recv = [torch.zeros(n * count, dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
            plan = ar.Plan(n, count, dtype, coll="allgather", **cfg)
            plan.run_oop(send, recv)
            torch.cuda.synchronize()
            want = x.reshape(-1).view(np.uint32) if dtype == "f32" else x.reshape(-1)
            for r in range(n):
                assert np.array_equal(to_bits(recv[r], dtype), want), (cfg, dtype)
            plan.destroy()


def test_collectives_full_size(ar):
    """128 MiB per rank: ReduceScatter of a 128 MiB send buffer and AllGather
    into a 128 MiB receive buffer (the paper's AllGather size), ring and
    direct, compared on the device."""
    import torch

    n = 8
    count = (128 << 20) // 4 // n
    x = workloads.draw(n, n * count, "f32", "uniform", workloads.SEED_BASE + 50)
    want = torch.from_numpy(ro.reduce_scatter(x, "f32")).to("cuda:0")
    send = to_device(x, "f32")
    for cfg in (dict(proto="simple", nchannels=32), dict(algo="direct")):
        say(f"RS full {cfg}")
        recv = [torch.empty(count, device="cuda:0") for _ in range(n)]
        plan = ar.Plan(n, count, "f32", coll="reducescatter", **cfg)
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        for r in range(n):
            assert torch.equal(recv[r].view(torch.int32), want[r].view(torch.int32)), (cfg, r)
        plan.destroy()
    del send
    xa = workloads.draw(n, count, "f32", "uniform", workloads.SEED_BASE + 51)
    want = torch.from_numpy(ro.all_gather(xa)).to("cuda:0")
    send = to_device(xa, "f32")
    for cfg in (dict(proto="simple", nchannels=32), dict(algo="direct")):
        say(f"AG full {cfg}")
        recv = [torch.empty(n * count, device="cuda:0") for _ in range(n)]
        plan = ar.Plan(n, count, "f32", coll="allgather", **cfg)
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        for r in range(n):
            assert torch.equal(recv[r].view(torch.int32), want.view(torch.int32)), (cfg, r)
        plan.destroy()


def test_collective_argument_errors(ar):
    import ctypes

    import torch

    n, count = 4, 64
    plan = ar.Plan(n, count, "f32", coll="reducescatter", proto="simple")
    send = [torch.zeros(n * count, device="cuda:0") for _ in range(n)]
    # recv of rank 1 inside rank 0's send buffer (not the in-place slot)
    recv = [send[0][count:2 * count], torch.zeros(count, device="cuda:0"), torch.zeros(count, device="cuda:0"),
            torch.zeros(count, device="cuda:0")]
    s = (ctypes.c_void_p * n)(*[t.data_ptr() for t in send])
    r = (ctypes.c_void_p * n)(*[t.data_ptr() for t in recv])
    assert ar.lib().ar_run_oop(plan.handle, s, r, None) == ar.AR_ERR_ARG
    plan.destroy()
    # a count that would misalign the blocks is refused
    h = ar.lib().ar_plan_ex(ctypes.byref(ar.make_desc(4, 6, "f32", "simple", 1, coll="allgather")))
    assert not h and ar.ar_last_error() == ar.AR_ERR_UNSUPPORTED
