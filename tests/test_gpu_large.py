"""Segments beyond 4 GiB: two ranks of 8 GiB of fp32 each, so a segment is
larger than a 32-bit byte offset can address.  Values are integers below
2^11 (every sum exact), periodic with two coprime periods that do not divide
2^30, so an access at the wrong element shows up as a wrong value.  The
result is checked on the device, slice by slice, against the sums written
out from the definition."""
from __future__ import annotations

import pytest

from tests.gpu_helpers import say

pytestmark = pytest.mark.gpu

P0, P1 = 1023, 1021          # 2^30 mod P != 0 for both periods
SLICE = 1 << 27              # elements per fill / check slice


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


def _pattern(lo, hi, period, scale):
    import torch

    i = torch.arange(lo, hi, dtype=torch.int64, device="cuda:0")
    return ((i % period) * scale).to(torch.float32)


def _fill(t, period, scale, offset=0):
    for lo in range(0, t.numel(), SLICE):
        hi = min(lo + SLICE, t.numel())
        t[lo:hi] = _pattern(offset + lo, offset + hi, period, scale)


def _check(t, label, offset=0):
    """t[k] == (offset + k) % P0 + 2 * ((offset + k) % P1) for every k."""
    import torch

    for lo in range(0, t.numel(), SLICE):
        hi = min(lo + SLICE, t.numel())
        want = _pattern(offset + lo, offset + hi, P0, 1) + _pattern(offset + lo, offset + hi, P1, 2)
        if not torch.equal(t[lo:hi], want):
            bad = int(torch.nonzero(t[lo:hi] != want)[0]) + lo
            raise AssertionError(f"{label}: element {bad} is {float(t[bad])}, want {float(want[bad - lo])}")


@pytest.mark.parametrize("cfg", [dict(algo="direct"), dict(proto="simple", nchannels=32)],
                         ids=["direct", "ring-simple"])
def test_allreduce_segment_beyond_4gib(ar, cfg):
    import torch

    n, count = 2, (1 << 31) + 3     # segments of 2^30 + 4 and 2^30 - 1 elements
    label = f"AllReduce N={n} count={count} f32 {cfg}"
    say(label)
    bufs = [torch.empty(count, dtype=torch.float32, device="cuda:0") for _ in range(n)]
    _fill(bufs[0], P0, 1)
    _fill(bufs[1], P1, 2)
    torch.cuda.synchronize()
    plan = ar.Plan(n, count, "f32", **cfg)
    assert plan.info["seg_elems"] * 4 > (1 << 32)
    plan.run(bufs)
    torch.cuda.synchronize()
    assert plan.status() == ar.AR_OK
    plan.destroy()
    for r in range(n):
        _check(bufs[r], f"{label} rank {r}")
    del bufs
    torch.cuda.empty_cache()


def test_allgather_block_beyond_4gib(ar):
    import torch

    n, count = 2, (1 << 30) + 8     # one block: 4 GiB + 32 bytes
    label = f"AllGather N={n} count={count} f32 direct"
    say(label)
    send = [torch.empty(count, dtype=torch.float32, device="cuda:0") for _ in range(n)]
    # block r holds the sum pattern of its own element range, so every
    # gathered buffer must read as one continuous pattern
    for r in range(n):
        for lo in range(0, count, SLICE):
            hi = min(lo + SLICE, count)
            off = r * count
            send[r][lo:hi] = _pattern(off + lo, off + hi, P0, 1) + _pattern(off + lo, off + hi, P1, 2)
    recv = [torch.empty(n * count, dtype=torch.float32, device="cuda:0") for _ in range(n)]
    torch.cuda.synchronize()
    plan = ar.Plan(n, count, "f32", coll="allgather", algo="direct")
    plan.run_oop(send, recv)
    torch.cuda.synchronize()
    assert plan.status() == ar.AR_OK
    plan.destroy()
    del send
    for r in range(n):
        _check(recv[r], f"{label} rank {r}")
    del recv
    torch.cuda.empty_cache()


def test_one_rank_copies(ar):
    """One rank: every collective is a copy of its one block, out of place;
    small and ragged sizes (tail bytes) and a copy over two 1 GiB windows."""
    import torch

    cases = [(c, dt) for c in (1, 3, 4, 5, 8, 12345) for dt in ("f32", "bf16")] + [((1 << 28) + 3, "f32")]
    for count, dtype in cases:
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        for coll in ("allreduce", "reducescatter", "allgather"):
            if coll != "allreduce" and count % (4 if dtype == "f32" else 8):
                continue
            label = f"one rank {coll} count={count} {dtype}"
            say(label)
            src = torch.randn(count, device="cuda:0").to(tdt)
            dst = torch.full((count,), float("nan"), device="cuda:0").to(tdt)
            plan = ar.Plan(1, count, dtype, coll=coll)
            plan.run_oop([src], [dst])
            torch.cuda.synchronize()
            assert plan.status() == ar.AR_OK
            plan.destroy()
            assert torch.equal(src.view(torch.int16 if dtype == "bf16" else torch.int32),
                               dst.view(torch.int16 if dtype == "bf16" else torch.int32)), label
            del src, dst
    torch.cuda.empty_cache()
