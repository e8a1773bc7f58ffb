"""Torn / stale line detector for the flag-in-line protocols (LL, LL128) and
the per-step trace of the debug kernel builds.

With AR_DEBUG_CHECK_LINES every writer fills each data word of a line with a
check word derived from that message's flag and the word's byte offset, and
every reader, once its normal protocol code has accepted a line by the
line's flag, compares each data word with the check word the flag implies.
A line whose data was left by another message (stale) or belongs elsewhere
(misplaced), or whose data and flag halves came from different writes
(torn), counts as bad.  Every case must report lines checked, and none bad.
The runs' outputs are undefined in this mode and are not compared."""
from __future__ import annotations

import numpy as np
import pytest

from tests.gpu_helpers import draw, say, to_device

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


def _run_checked(ar, n, count, dtype, coll, runs, debug, **cfg):
    import torch

    a = 4 if dtype == "f32" else 8
    send_n = count * n if coll == "reducescatter" else count
    recv_n = count * n if coll == "allgather" else count
    if coll == "allreduce":
        send_n = recv_n = count
    assert coll == "allreduce" or count % a == 0
    x = draw(n, send_n, dtype, "uniform", seed=count + 7 * n)
    send = to_device(x, dtype)
    recv = [torch.empty(recv_n, dtype=send[0].dtype, device="cuda:0") for _ in range(n)]
    plan = ar.Plan(n, count, dtype, coll=coll, debug_flags=debug, **cfg)
    label = f"line check N={n} count={count} {dtype} {coll} runs={runs} debug={debug} {cfg}"
    say(label)
    try:
        for _ in range(runs):
            plan.run_oop(send, recv)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK, label
        st = plan.debug_stats()
        info = plan.info
    finally:
        plan.destroy()
    say(f"  {st}")
    assert st["lines_bad"] == 0, (label, st)
    assert st["lines_first_read"] <= st["lines_checked"]
    # every line that crossed a link was checked once: about the wire bytes
    # per run over the line size (ragged message ends add a few lines)
    line = 8 if info["proto"] == ar.AR_PROTO_LL else 128
    wire = info["wire_bytes_per_run"]
    if info["peer_direct"] and coll != "allgather":
        # the chain starts' peer reads cross a link without line flags (a
        # two-rank ReduceScatter then moves no line at all)
        wire -= (count if coll == "allreduce" else n * count) * (4 if dtype == "f32" else 2)
    approx = wire * runs / line
    assert st["lines_checked"] > 0 or approx == 0, (label, st)
    assert 0.95 * approx <= st["lines_checked"] <= 1.25 * approx + 64 * runs * info["grid"], (label, st, approx)
    return st


@pytest.mark.parametrize("proto", ("ll", "ll128"))
@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_line_check_collectives(ar, proto, dtype):
    """Every collective and rank count, ragged counts, one and three
    channels, a few runs each on one plan (lines of earlier runs stay in
    the slots and must never be accepted for later messages)."""
    a = 4 if dtype == "f32" else 8
    dbg = ar.AR_DEBUG_CHECK_LINES
    # also with every hop through the FIFOs (by default the reduction chains
    # start with a peer read)
    modes = (0, ar.AR_PLAN_FIFO_ONLY)
    for n in (2, 3, 8):
        for flags in modes:
            for count, nch in ((1000 * a + 3, 1), (4099, 3), (24 * a, 2)):
                _run_checked(ar, n, count, dtype, "allreduce", 4, dbg, proto=proto, nchannels=nch, flags=flags)
            for coll in ("reducescatter", "allgather"):
                _run_checked(ar, n, 500 * a, dtype, coll, 3, dbg, proto=proto, nchannels=2, flags=flags)
    # a depth-2 FIFO with one channel and one wave: slots are reused every
    # other message
    _run_checked(ar, 8, 3000 * a, dtype, "allreduce", 8, dbg, proto=proto, nchannels=1, nwaves=1, fifo_depth=2)


@pytest.mark.parametrize("proto", ("ll", "ll128"))
@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_line_check_stress(ar, proto, dtype):
    """Many channels and waves, 4 MiB per rank, repeated runs, with and
    without jittered posts: tens of millions of lines accepted while their
    writers are still writing neighbouring lines.  For LL128 both ways of
    accepting a batch are exercised: from the first load of its lines, and
    from a re-read after its flags were seen current."""
    e = 4 if dtype == "f32" else 2
    count = (4 << 20) // e
    dbg = ar.AR_DEBUG_CHECK_LINES
    st1 = _run_checked(ar, 8, count, dtype, "allreduce", 30, dbg, proto=proto, nchannels=32)
    st2 = _run_checked(ar, 8, count, dtype, "allreduce", 10, dbg | ar.AR_DEBUG_JITTER, proto=proto, nchannels=16,
                       nwaves=8)
    st3 = _run_checked(ar, 8, count // 16, dtype, "allreduce", 200, dbg, proto=proto, nchannels=4, nwaves=1)
    total = sum(s["lines_checked"] for s in (st1, st2, st3))
    first = sum(s["lines_first_read"] for s in (st1, st2, st3))
    say(f"{proto} {dtype}: {total} lines checked, {first} accepted on the first load, 0 bad")
    assert first > 0 and first < total


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_line_check_ll128_ordered(ar, dtype):
    """With AR_PLAN_LL128_ORDERED no line is taken from a load that also
    brought its flag: the checker counts no first-load acceptances, and no
    bad line."""
    e = 4 if dtype == "f32" else 2
    dbg = ar.AR_DEBUG_CHECK_LINES
    for count, ch, w, runs in (((4 << 20) // e, 32, 4, 10), (5000, 1, 1, 20), ((1 << 20) // e, 4, 1, 20)):
        st = _run_checked(ar, 8, count, dtype, "allreduce", runs, dbg, proto="ll128", nchannels=ch, nwaves=w,
                          flags=ar.AR_PLAN_LL128_ORDERED)
        assert st["lines_first_read"] == 0, st


def test_trace_records(ar):
    """AR_DEBUG_TRACE: one record per ring step of channel 0 / wave 0 of
    every rank.  Stamps inside a step are ordered; message indices advance
    by one per step; and, across ranks, the step that takes a message
    accepts it after its sender finished the stores that publish it (the
    100 MHz real-time counter is common to every XCD)."""
    import torch

    n, count = 8, 8 * 4096
    for proto in ("simple", "ll", "ll128"):
        plan = ar.Plan(n, count, "f32", proto=proto, nchannels=2, nwaves=1, debug_flags=ar.AR_DEBUG_TRACE,
                       flags=ar.AR_PLAN_FIFO_ONLY)
        per_rank = 64
        buf = torch.zeros(n * per_rank * 8, dtype=torch.int64, device="cuda:0")
        plan.set_trace(buf)
        x = draw(n, count, "f32", "uniform", seed=3)
        send = to_device(x, "f32")
        recv = [torch.empty_like(t) for t in send]
        say(f"trace {proto}")
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK
        nsteps = plan.info["nchunks"] * (2 * n - 1)
        plan.destroy()
        rec = buf.cpu().numpy().view(np.uint64).reshape(n, per_rank, 8)
        t_begin, t_recv, polls, t_issued, t_drained, t_posted, msg, kind = (rec[:, :nsteps, i] for i in range(8))
        assert np.all(rec[:, nsteps:] == 0)
        assert np.all(t_begin > 0)
        for r in range(n):
            # message indices: the send steps of a run are consecutive
            sends = msg[r][kind[r] != 4]  # kind 4: receive-only (recvCopy)
            assert np.all(np.diff(sends.astype(np.int64)) == 1), (proto, r, sends)
            for k in range(nsteps):
                stamps = [v for v in (t_begin[r, k], t_recv[r, k], t_issued[r, k], t_drained[r, k], t_posted[r, k])
                          if v]
                assert stamps == sorted(stamps), (proto, r, k, stamps)
        # causality across ranks: rank r+1's step k+1 takes the message rank
        # r published in its step k
        for r in range(n):
            q = (r + 1) % n
            for k in range(nsteps - 1):
                if k % (2 * n - 1) == 2 * n - 2:
                    continue  # the last step of a chunk sends nothing
                pub = t_drained[r, k] if proto != "ll" else t_begin[r, k]
                assert t_recv[q, k + 1] >= pub, (proto, r, k, int(t_recv[q, k + 1]), int(pub))
