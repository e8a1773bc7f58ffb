"""The allocation-free entry point (ar_run_noalloc) against the plan-based one
(ar_plan_ex + ar_run_oop), through the C ABI, bit for bit, and both against
the CPU oracle.  Each case calls the allocation-free entry twice in a row on
the same device scratch, the second time with a smaller input, so the second
call must clear what the first one left there."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import ring_oracle as ro
from tests.gpu_helpers import draw, say, to_bits, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


def _oracle(x, dtype, coll):
    if coll == "allreduce":
        y = ro.allreduce(x, dtype)
        return np.stack([y] * x.shape[0])
    if coll == "reducescatter":
        return ro.reduce_scatter(x, dtype)
    y = ro.all_gather(x)
    return np.stack([y] * x.shape[0])


def _bits(ts, dtype):
    return np.stack([to_bits(t, dtype) for t in ts])


def _one(ar, n, count, dtype, coll, cfg, seed):
    """Run one collective both ways (out of place) and return both results."""
    import torch

    send_count = count * n if coll == "reducescatter" else count
    recv_count = count * n if coll == "allgather" else count
    if coll == "allreduce":
        send_count = recv_count = count
    x = draw(n, send_count, dtype, "normal", seed)
    send = to_device(x, dtype)
    recv_a = [torch.full((recv_count,), float("nan"), dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
    recv_b = [torch.full((recv_count,), float("nan"), dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
    say(f"noalloc N={n} count={count} {dtype} {coll} {cfg}")
    ar.run_noalloc(send, recv_a, coll=coll, **cfg)
    torch.cuda.synchronize()
    plan = ar.Plan(n, count, dtype, coll=coll, **cfg)
    try:
        plan.run_oop(send, recv_b)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        info = plan.info
    finally:
        plan.destroy()
    want = _oracle(x, dtype, coll)
    want = want.view(np.uint32) if dtype == "f32" else want
    a, b = _bits(recv_a, dtype), _bits(recv_b, dtype)
    assert np.array_equal(a, b), f"noalloc differs from ar_run_oop: {cfg}"
    assert np.array_equal(a.reshape(want.shape), want), f"noalloc differs from the oracle: {cfg}"
    return info


CASES = [
    ("allreduce", "f32", dict(proto="simple", nchannels=4)),
    ("allreduce", "f32", dict(proto="simple", nchannels=3, chunk_bytes=512, flags=2)),
    ("allreduce", "f32", dict(proto="ll", nchannels=2)),
    ("allreduce", "f32", dict(proto="ll128", nchannels=2)),
    ("allreduce", "bf16", dict(proto="simple", nchannels=5)),
    ("allreduce", "bf16", dict(proto="ll", nchannels=3)),
    ("allreduce", "bf16", dict(proto="ll128", nchannels=1)),
    ("allreduce", "f32", dict(algo="direct")),
    ("allreduce", "f32", dict(proto="auto")),
    ("reducescatter", "f32", dict(proto="ll", nchannels=2)),
    ("reducescatter", "bf16", dict(proto="simple", nchannels=2)),
    ("allgather", "f32", dict(proto="ll128", nchannels=2)),
    ("allgather", "bf16", dict(proto="simple", nchannels=3)),
]


@pytest.mark.parametrize("coll,dtype,cfg", CASES, ids=[f"{c}-{d}-{i}" for i, (c, d, _) in enumerate(CASES)])
def test_noalloc_matches_plan_twice(ar, coll, dtype, cfg):
    a = 4 if dtype == "f32" else 8
    # first a larger call, then a smaller one on the same scratch
    for n, count in ((8, 6000 * a), (3, 37 * a)):
        info = _one(ar, n, count if coll != "allreduce" else count + 3, dtype, coll, cfg, seed=count + n)
        if info["algo"] == ar.AR_ALGO_RING:
            assert info["fifo_bytes"] + info["flag_bytes"] <= ar.AR_NOALLOC_SCRATCH_BYTES


def test_noalloc_in_place_and_ranks(ar):
    """In place, N from 1 to 16, ragged counts, on the scratch left by the
    cases before."""
    import torch

    for n, count, proto in ((1, 1001, "simple"), (2, 5, "ll"), (5, 777, "ll128"), (16, 4099, "simple"),
                            (8, 1, "ll"), (8, 0, "simple")):
        x = draw(n, count, "f32", "uniform", seed=31 * n + count)
        ts = to_device(x, "f32")
        say(f"noalloc in place N={n} count={count} {proto}")
        ar.run_noalloc(ts, proto=proto, nchannels=2)
        torch.cuda.synchronize()
        want = ro.allreduce(x, "f32").view(np.uint32)
        for t in ts:
            assert np.array_equal(to_bits(t, "f32"), want)


def test_noalloc_rejects_what_it_cannot_hold(ar):
    """Requests beyond the static scratch, and profiling (which needs
    events), are refused on the host before anything is launched."""
    import torch

    n, count = 8, 1 << 20
    ts = [torch.zeros(count, dtype=torch.float32, device="cuda:0") for _ in range(n)]
    # LL, 2 channels x 16 waves x 8 ranks x 4 slots of 32 KiB: 32 MiB of FIFO
    big = dict(proto="ll", nchannels=2, nwaves=16, chunk_bytes=4 << 20)
    with pytest.raises(ar.ARError) as e:
        ar.run_noalloc(ts, **big)
    assert e.value.code == ar.AR_ERR_SCRATCH
    with pytest.raises(ar.ARError) as e:
        ar.run_noalloc(ts, proto="simple", nchannels=2, flags=ar.AR_PLAN_PROFILE)
    assert e.value.code == ar.AR_ERR_UNSUPPORTED
    desc = ar.make_desc(n, count, "f32", **big)
    g = ar.ar_plan_geometry(desc)
    assert g["fifo_bytes"] > ar.AR_NOALLOC_SCRATCH_BYTES
    torch.cuda.synchronize()


@pytest.mark.parametrize("cfg", [dict(proto="ll", nchannels=2), dict(proto="simple", nchannels=3),
                                 dict(proto="ll128", nchannels=2)], ids=lambda c: c["proto"])
def test_noalloc_graph_replay(ar, cfg):
    """Calls captured into a HIP graph: each replay clears the scratch with
    the captured fill kernel and runs the ring from message 0 again, so
    every replay, on fresh input values, gives the oracle's bits; eager
    calls with other values run between the replays."""
    import torch

    n, count = 8, 4099
    x0 = draw(n, count, "f32", "normal", seed=810)
    send = to_device(x0, "f32")
    recv = [torch.full((count,), float("nan"), device="cuda:0") for _ in range(n)]
    ar.run_noalloc(send, recv, **cfg)  # eager first (the device's scratch address is looked up here)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(recv, "f32"), _oracle(x0, "f32", "allreduce").view(np.uint32))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ar.run_noalloc(send, recv, stream=side, **cfg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for _ in range(2):
            ar.run_noalloc(send, recv, stream=side, **cfg)
    torch.cuda.synchronize()
    for rep in range(4):
        say(f"noalloc graph {cfg} replay {rep}")
        x = draw(n, count, "f32", "normal", seed=820 + rep)
        host = to_device(x, "f32")
        for r in range(n):
            send[r].copy_(host[r])
            recv[r].fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_bits(recv, "f32"), _oracle(x, "f32", "allreduce").view(np.uint32)), rep
        x2 = draw(n, count, "f32", "normal", seed=830 + rep)
        host = to_device(x2, "f32")
        for r in range(n):
            send[r].copy_(host[r])
        ar.run_noalloc(send, recv, **cfg)
        torch.cuda.synchronize()
        assert np.array_equal(_bits(recv, "f32"), _oracle(x2, "f32", "allreduce").view(np.uint32)), rep
    del g
