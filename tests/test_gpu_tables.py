"""GPU parity of every row of the built-in tuner tables at its own size.

The fp32 AllReduce rows are covered by the D4 sweep in test_gpu_parity.py.
Here: the bf16 AllReduce table, and the ReduceScatter and AllGather tables
of both data types, at every power-of-two size from 4 KiB to 128 MiB
(AllReduce: bytes per rank; ReduceScatter and AllGather: bytes of one
rank's full buffer).  Each size runs the table's overall choice and its
ring choice (protocol, channels, chunk and waves for that size), out of
place, and compares every rank's output with the CPU oracle bit for bit.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads
from oracle import ring_oracle as ro
from tests.gpu_helpers import say, to_device

pytestmark = pytest.mark.gpu

N = 8
SIZES = workloads.WORKLOADS["D4"].extra["sizes"]
CFGS = (dict(proto="auto"), dict(proto="auto", algo="ring"))
ELEM = {"f32": 4, "bf16": 2}


@pytest.fixture(scope="module")
def ar():
    import torch

    import paper_2603_11438_amd as ar

    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    ar.lib()
    ar.ar_set_tuner(None)
    return ar


def _on_device(bits: np.ndarray, dtype: str):
    """A 1-D array of result bits as a device tensor of the data type."""
    return to_device(bits[None, :].view(np.float32 if dtype == "f32" else np.uint16), dtype)[0]


def _same(t, want_dev, dtype, label):
    import torch

    iv = torch.int32 if dtype == "f32" else torch.int16
    if not torch.equal(t.view(iv), want_dev.view(iv)):
        bad = (t.view(iv) != want_dev.view(iv)).nonzero()
        raise AssertionError(f"{label}: {bad.numel()} elements differ, first {int(bad[0])}")


def _bits(y: np.ndarray, dtype: str) -> np.ndarray:
    return y.view(np.uint32) if dtype == "f32" else y


def _tag(info) -> str:
    return f"[{info['algo_name']}/{info['proto_name']}/{info['nchannels']}]"


def _run(ar, coll, count, dtype, cfg, send, recv_elems):
    import torch

    recv = [torch.empty(recv_elems, dtype=send[0].dtype, device="cuda:0") for _ in range(N)]
    plan = ar.Plan(N, count, dtype, coll=coll, **cfg)
    try:
        plan.run_oop(send, recv)
        torch.cuda.synchronize()
        assert plan.status() == ar.AR_OK, (coll, count, dtype, cfg)
        return recv, dict(plan.info)
    finally:
        plan.destroy()


def test_allreduce_bf16_table_rows(ar):
    for size in SIZES:
        count = size // 2
        x = workloads.draw(N, count, "bf16", "normal", workloads.SEED_BASE + 60)
        want = _on_device(ro.allreduce_bf16(x), "bf16")
        send = to_device(x, "bf16")
        del x
        for cfg in CFGS:
            label = f"AllReduce bf16 {size} B {cfg}"
            say(label)
            recv, info = _run(ar, "allreduce", count, "bf16", cfg, send, count)
            for r in range(N):
                _same(recv[r], want, "bf16", f"{label} {_tag(info)} rank {r}")


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_reduce_scatter_table_rows(ar, dtype):
    for size in SIZES:
        count = size // ELEM[dtype] // N  # elements of one block
        x = workloads.draw(N, N * count, dtype, "uniform", workloads.SEED_BASE + 61)
        want = to_device(_bits(ro.reduce_scatter(x, dtype), dtype).view(np.float32 if dtype == "f32" else np.uint16),
                         dtype)
        send = to_device(x, dtype)
        del x
        for cfg in CFGS:
            label = f"ReduceScatter {dtype} {size} B {cfg}"
            say(label)
            recv, info = _run(ar, "reducescatter", count, dtype, cfg, send, count)
            for r in range(N):
                _same(recv[r], want[r], dtype, f"{label} {_tag(info)} rank {r}")


@pytest.mark.parametrize("dtype", ("f32", "bf16"))
def test_all_gather_table_rows(ar, dtype):
    for size in SIZES:
        count = size // ELEM[dtype] // N  # elements each rank contributes
        x = workloads.draw(N, count, dtype, "uniform", workloads.SEED_BASE + 62)
        want = _on_device(_bits(ro.all_gather(x), dtype), dtype)
        send = to_device(x, dtype)
        del x
        for cfg in CFGS:
            label = f"AllGather {dtype} {size} B {cfg}"
            say(label)
            recv, info = _run(ar, "allgather", count, dtype, cfg, send, N * count)
            for r in range(N):
                _same(recv[r], want, dtype, f"{label} {_tag(info)} rank {r}")
