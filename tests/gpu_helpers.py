"""Helpers shared by the GPU tests: move seeded inputs to the device, run
the HIP AllReduce through the C ABI binding, and compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np

import workloads
from oracle import ring_oracle as ro


def say(*a):
    """Print and flush, so a log names the case even if the process dies."""
    print(*a, flush=True)
    sys.stdout.flush()


def to_device(x: np.ndarray, dtype: str):
    """One separately allocated device tensor per rank (each 16-byte aligned)."""
    import torch

    n = x.shape[0]
    if dtype == "f32":
        return [torch.from_numpy(np.ascontiguousarray(x[r])).to("cuda:0") for r in range(n)]
    return [torch.from_numpy(np.ascontiguousarray(x[r]).view(np.int16)).view(torch.bfloat16).to("cuda:0")
            for r in range(n)]


def to_bits(t, dtype: str) -> np.ndarray:
    import torch

    c = t.detach().cpu()
    if dtype == "f32":
        return c.view(torch.int32).numpy().view(np.uint32)
    return c.view(torch.int16).numpy().view(np.uint16)


def oracle_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return ro.allreduce_f32(x).view(np.uint32)
    return ro.allreduce_bf16(x)


def assert_ranks_equal(ts, want: np.ndarray, dtype: str, label: str = ""):
    for r, t in enumerate(ts):
        got = to_bits(t, dtype)
        if not np.array_equal(got, want):
            bad = np.flatnonzero(got != want)
            i = int(bad[0])
            raise AssertionError(f"{label}: rank {r}: {bad.size} elements differ, first at {i}: "
                                 f"got {got[i]:#x} want {want[i]:#x}")


def run_case(ar, x: np.ndarray, dtype: str, label: str = "", poison: bool = False, **plan_kw):
    """Run one AllReduce of x (N, count) and assert every rank equals the oracle."""
    import torch

    n, count = x.shape
    say(f"case {label}: N={n} count={count} dtype={dtype} {plan_kw}")
    ts = to_device(x, dtype)
    want = oracle_bits(x, dtype)
    plan = ar.Plan(n, count, dtype, **plan_kw)
    try:
        if poison:
            plan.poison()
        plan.run(ts)
        torch.cuda.synchronize()
        st = plan.status()
        assert st == ar.AR_OK, f"{label}: status {ar.ar_strerror(st)}"
        assert_ranks_equal(ts, want, dtype, label)
        return plan.info
    finally:
        plan.destroy()


def draw(n, count, dtype, dist="uniform", seed=0):
    return workloads.draw(n, count, dtype, dist, seed)
