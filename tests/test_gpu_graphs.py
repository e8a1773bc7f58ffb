"""HIP-graph capture and replay of the collectives, checked against eager
runs and the oracle on every replay.

The ring keeps its message epoch in device memory, so a captured launch
continues the flag counters of the runs before it.  Each replay here gets
fresh input values (copied into the captured send buffers), so a replay
that read stale FIFO contents or stale counters would produce the previous
input's sums and fail.  Eager runs and synchronisations sit between the
replays, as a real program's would."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import ring_oracle as ro
from tests.gpu_helpers import assert_ranks_equal, draw, oracle_bits, say, to_bits, to_device

pytestmark = pytest.mark.gpu

CFGS = [dict(proto="simple", nchannels=2), dict(proto="ll", nchannels=2), dict(proto="ll128", nchannels=2),
        dict(proto="simple", nchannels=1, chunk_bytes=1024, fifo_depth=2), dict(algo="direct")]


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


def _want(coll, x, dtype, n):
    if coll == "allreduce":
        y = ro.allreduce(x, dtype)
        y = y.view(np.uint32) if dtype == "f32" else y
        return np.stack([y] * n)
    if coll == "reducescatter":
        y = ro.reduce_scatter(x, dtype)
        return y.view(np.uint32) if dtype == "f32" else y
    y = ro.all_gather(x)
    y = y.view(np.uint32) if dtype == "f32" else y
    return np.stack([y] * n)


def _shapes(coll, n, count):
    """(elements per send buffer, elements per recv buffer)."""
    if coll == "allreduce":
        return count, count
    if coll == "reducescatter":
        return n * count, count
    return count, n * count


def _got(recv, dtype):
    return np.stack([to_bits(t, dtype) for t in recv])


def _graph_case(ar, coll, dtype, cfg, n, count, runs_per_graph=3, replays=4):
    import torch

    ns, nr = _shapes(coll, n, count)
    label = f"graph {coll} {dtype} N={n} count={count} {cfg}"
    say(label)
    plan = ar.Plan(n, count, dtype, coll=coll, **cfg)
    x0 = draw(n, ns, dtype, "normal", seed=500 + count)
    send = to_device(x0, dtype)
    recv = [torch.full((nr,), float("nan"), device="cuda:0").to(send[0].dtype) for _ in range(n)]

    # eager reference run
    plan.run_oop(send, recv)
    torch.cuda.synchronize()
    assert plan.status() == ar.AR_OK
    assert np.array_equal(_got(recv, dtype), _want(coll, x0, dtype, n)), f"{label}: eager"

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        plan.run_oop(send, recv, side)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for _ in range(runs_per_graph):
            plan.run_oop(send, recv, side)
    torch.cuda.synchronize()

    for rep in range(replays):
        x = draw(n, ns, dtype, "normal", seed=600 + 10 * rep + count)
        host = to_device(x, dtype)
        for r in range(n):
            send[r].copy_(host[r])
            recv[r].fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK, f"{label}: replay {rep} status"
        assert np.array_equal(_got(recv, dtype), _want(coll, x, dtype, n)), f"{label}: replay {rep}"
        # the program's own eager work between replays, on new values again
        x2 = draw(n, ns, dtype, "normal", seed=700 + 10 * rep + count)
        host = to_device(x2, dtype)
        for r in range(n):
            send[r].copy_(host[r])
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        assert np.array_equal(_got(recv, dtype), _want(coll, x2, dtype, n)), f"{label}: eager after {rep}"
    del g
    plan.destroy()


@pytest.mark.parametrize("cfg", CFGS, ids=lambda c: "-".join(f"{k}{v}" for k, v in c.items()))
def test_graph_replay_allreduce(ar, cfg):
    _graph_case(ar, "allreduce", "f32", cfg, 8, 4099)
    _graph_case(ar, "allreduce", "bf16", cfg, 3, 1000)


@pytest.mark.parametrize("coll", ("reducescatter", "allgather"))
@pytest.mark.parametrize("cfg", CFGS[:2] + CFGS[4:], ids=lambda c: "-".join(f"{k}{v}" for k, v in c.items()))
def test_graph_replay_reduce_scatter_all_gather(ar, coll, cfg):
    _graph_case(ar, coll, "f32", cfg, 8, 1024)


def test_epoch_continues_across_many_runs(ar):
    """More LL messages than FIFO slots across eager runs, replays and a
    second plan sharing nothing: the device-side epoch keeps every run's
    flags distinct from the stale lines left in the slots."""
    import torch

    n, count = 4, 64
    plan = ar.Plan(n, count, "f32", proto="ll", nchannels=1, nwaves=1, fifo_depth=2)
    x = draw(n, count, "f32", "normal", seed=77)
    want = ro.allreduce_f32(x).view(np.uint32)
    send = to_device(x, "f32")
    recv = [torch.empty(count, device="cuda:0") for _ in range(n)]
    for i in range(257):
        plan.run_oop(send, recv)
    torch.cuda.synchronize()
    assert plan.status() == ar.AR_OK
    for r in range(n):
        assert np.array_equal(to_bits(recv[r], "f32"), want)
    plan.destroy()


def test_ring_plans_on_several_streams(ar):
    """Ring plans of different protocols launched alternately on three
    streams (each grid small enough that all fit at once, so nothing here
    depends on the ordering to finish), with the direct algorithm on a
    fourth: the library orders the ring launches across streams, and every
    result matches the oracle."""
    import torch

    n = 8
    streams = [torch.cuda.Stream() for _ in range(4)]
    specs = [(50000, dict(proto="simple", nchannels=4)), (30001, dict(proto="ll", nchannels=2)),
             (20011, dict(proto="ll128", nchannels=2)), (40000, dict(algo="direct"))]
    plans, xs, sends, recvs = [], [], [], []
    for i, (count, cfg) in enumerate(specs):
        x = draw(n, count, "f32", "uniform", seed=60 + i)
        xs.append(x)
        plans.append(ar.Plan(n, count, "f32", **cfg))
        sends.append(to_device(x, "f32"))
    torch.cuda.synchronize()
    for rep in range(12):
        say(f"several streams, round {rep}")
        rounds = []
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                recv = [torch.full_like(t, float("nan")) for t in sends[i]]
                plans[i].run_oop(sends[i], recv, stream=s)
                rounds.append(recv)
        torch.cuda.synchronize()
        for i in range(len(specs)):
            assert plans[i].status() == ar.AR_OK
            assert_ranks_equal(rounds[i], oracle_bits(xs[i], "f32"), "f32", f"stream {i} round {rep}")
    for p in plans:
        p.destroy()


def test_ring_plans_from_two_host_threads(ar):
    """Two host threads, each with its own ring plan and stream, launch 40
    runs each at the same time (the C calls run concurrently: ctypes
    releases the interpreter lock).  The launch gate's per-device lock and
    event keep the sequence consistent; every run's result is checked."""
    import threading

    import torch

    n = 8
    specs = [(30011, dict(proto="ll", nchannels=2)), (20000, dict(proto="simple", nchannels=3))]
    results, errors = {}, []

    def worker(i, count, cfg):
        try:
            torch.cuda.set_device(0)
            x = draw(n, count, "f32", "uniform", seed=90 + i)
            send = to_device(x, "f32")
            plan = ar.Plan(n, count, "f32", **cfg)
            stream = torch.cuda.Stream()
            fn_recv = [[torch.empty_like(t) for t in send] for _ in range(40)]
            with torch.cuda.stream(stream):
                for k in range(40):
                    plan.run_oop(send, fn_recv[k], stream=stream)
            stream.synchronize()
            results[i] = (plan.status(), x, fn_recv)
            plan.destroy()
        except Exception as e:  # reported below
            errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(i, c, cfg)) for i, (c, cfg) in enumerate(specs)]
    say("two host threads, two streams")
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    torch.cuda.synchronize()
    assert not errors, errors
    for i, (st, x, recvs) in results.items():
        assert st == ar.AR_OK
        want = oracle_bits(x, "f32")
        for k, recv in enumerate(recvs):
            assert_ranks_equal(recv, want, "f32", f"thread {i} run {k}")
