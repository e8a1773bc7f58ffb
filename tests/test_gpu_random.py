"""Randomised GPU parity: seeded random plans (collective, algorithm,
protocol, rank count, element count, dtype, channels, chunk, waves, FIFO
depth, placement, in place or not), each checked bit for bit against the
oracle, run twice on one plan (the second run on new values, so stale FIFO
contents or counters would show)."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import ring_oracle as ro
from tests.gpu_helpers import draw, say, to_bits, to_device

pytestmark = pytest.mark.gpu

NCASES = 200


def _case(rng):
    coll = rng.choice(["allreduce", "allreduce", "reducescatter", "allgather"])
    dtype = rng.choice(["f32", "bf16"])
    n = int(rng.choice([2, 3, 4, 5, 7, 8, 11, 16]))
    a = 4 if dtype == "f32" else 8
    if coll == "allreduce":
        count = int(rng.integers(1, 20000))
    else:
        count = a * int(rng.integers(1, 2000))
    algo = rng.choice(["ring", "ring", "ring", "direct"])
    cfg = {"algo": str(algo)}
    if algo == "ring":
        cfg["proto"] = str(rng.choice(["simple", "ll", "ll128"]))
        cfg["nchannels"] = int(rng.integers(1, 9))
        cfg["nwaves"] = int(rng.choice([1, 2, 4, 8]))
        cfg["chunk_bytes"] = int(rng.choice([16, 256, 1024, 4096, 65536]))
        cfg["fifo_depth"] = int(rng.choice([2, 3, 4, 8]))
        cfg["placement"] = int(rng.integers(0, 2))
        # 2: Simple all-gather through the FIFOs; 4: LL128 reads lines only
        # after their flags
        cfg["flags"] = int(rng.choice([0, 2, 4]))
    else:
        cfg["nchannels"] = int(rng.choice([0, 1, 3, 16]))
        cfg["nwaves"] = int(rng.choice([0, 1, 4, 16]))
        cfg["direct_unroll"] = int(rng.choice([0, 1, 2]))
    return str(coll), str(dtype), n, count, cfg, bool(rng.integers(0, 2))


def _bits(x, dtype):
    return x.view(np.uint32) if dtype == "f32" else x


def _expected(coll, x, dtype, n):
    if coll == "allreduce":
        return np.stack([_bits(ro.allreduce(x, dtype), dtype)] * n)
    if coll == "reducescatter":
        return _bits(ro.reduce_scatter(x, dtype), dtype)
    return np.stack([_bits(ro.all_gather(x), dtype)] * n)


def _run(ar, plan, coll, x, dtype, n, count, in_place):
    import torch

    if coll == "allreduce":
        if in_place:
            bufs = to_device(x, dtype)
            plan.run(bufs)
            torch.cuda.synchronize()
            return np.stack([to_bits(b, dtype) for b in bufs])
        send = to_device(x, dtype)
        recv = [torch.empty_like(t) for t in send]
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        return np.stack([to_bits(b, dtype) for b in recv])
    if coll == "reducescatter":
        send = to_device(x, dtype)
        if in_place:
            plan.run(send)
            torch.cuda.synchronize()
            return np.stack([to_bits(send[r], dtype)[r * count:(r + 1) * count] for r in range(n)])
        recv = [torch.empty(count, dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        return np.stack([to_bits(b, dtype) for b in recv])
    if in_place:
        full = np.zeros((n, n * count), dtype=x.dtype)
        for r in range(n):
            full[r, r * count:(r + 1) * count] = x[r]
        bufs = to_device(full, dtype)
        plan.run(bufs)
        torch.cuda.synchronize()
        return np.stack([to_bits(b, dtype) for b in bufs])
    send = to_device(x, dtype)
    recv = [torch.empty(n * count, dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
    plan.run_oop(send, recv)
    torch.cuda.synchronize()
    return np.stack([to_bits(b, dtype) for b in recv])


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


@pytest.mark.parametrize("block", range(4))
def test_random_plans(ar, block):
    rng = np.random.default_rng(20260 + block)
    for i in range(NCASES // 4):
        coll, dtype, n, count, cfg, in_place = _case(rng)
        label = f"random block {block} case {i}: {coll} {dtype} N={n} count={count} {cfg} in_place={in_place}"
        say(label)
        plan = ar.Plan(n, count, dtype, coll=coll, **cfg)
        try:
            for rep in range(2):
                elems = n * count if coll == "reducescatter" else count
                x = draw(n, elems, dtype, "normal", seed=1000 * block + 10 * i + rep)
                got = _run(ar, plan, coll, x, dtype, n, count, in_place)
                assert plan.status() == ar.AR_OK, f"{label}: status"
                assert np.array_equal(got, _expected(coll, x, dtype, n)), f"{label}: run {rep}"
        finally:
            plan.destroy()
