"""Seeded synthetic inputs for the simulated-ring AllReduce.

This module only draws numbers: it holds none of the reduction's
arithmetic, so both the CPU oracle (under ``oracle/``) and the HIP path
can take their inputs from it without sharing any of the method.

The paper measures AllReduce by message size on data-parallel gradient
buckets (section 5.3, Table 2 and Figure 2) and names no dataset, so the
workloads are synthetic: N rank buffers of ``count`` elements each, with
the value distributions below.

Every array is drawn with ``numpy.random.default_rng(seed)`` (PCG64) in
one call of shape (N, count), in float32.  bf16 inputs are the float32
draw converted by torch's CPU ``.to(torch.bfloat16)`` (a library
round-to-nearest-even), returned as raw uint16 bit patterns.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 11438

FP32 = "f32"
BF16 = "bf16"
ELEM_BYTES = {FP32: 4, BF16: 2}


def draw(nranks: int, count: int, dtype: str, dist: str, seed: int) -> np.ndarray:
    """Return an (nranks, count) array: float32 for "f32", uint16 bf16 bits for "bf16".

    dist is one of
      "int8"    integers drawn uniformly from {-8, ..., 8} inclusive,
      "uniform" float32 u in [0, 1) mapped to 2u - 1, i.e. [-1, 1),
      "normal"  standard normal N(0, 1) (gradient-like values),
      "ones"    every element 1.0 (no randomness).
    """
    if nranks < 0 or count < 0:
        raise ValueError("nranks and count must be non-negative")
    rng = np.random.default_rng(seed)
    shape = (nranks, count)
    if dist == "int8":
        a = rng.integers(-8, 9, size=shape, dtype=np.int32).astype(np.float32)
    elif dist == "uniform":
        a = rng.random(size=shape, dtype=np.float32)
        a *= np.float32(2.0)
        a -= np.float32(1.0)
    elif dist == "normal":
        a = rng.standard_normal(size=shape, dtype=np.float32)
    elif dist == "ones":
        a = np.ones(shape, dtype=np.float32)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    if dtype == FP32:
        return a
    if dtype == BF16:
        return to_bf16_bits_torch(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def to_bf16_bits_torch(a: np.ndarray) -> np.ndarray:
    """float32 array -> uint16 bf16 bit patterns via torch's CPU conversion."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


@dataclass(frozen=True)
class Workload:
    """One named synthetic workload: N ranks x count elements of dtype."""

    name: str
    nranks: int
    count: int
    dtype: str
    dist: str
    seed: int
    protos: tuple = ()
    channels: tuple = ()
    chunks: tuple = ()
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def bytes_per_rank(self) -> int:
        return self.count * ELEM_BYTES[self.dtype]

    def draw(self) -> np.ndarray:
        return draw(self.nranks, self.count, self.dtype, self.dist, self.seed)


KiB = 1024
MiB = 1024 * 1024

WORKLOADS = {
    # 8 ranks x 4 KiB fp32, integer-valued in [-8, 8]; Simple, 1 channel, 1 KiB chunk.
    "D1": Workload("D1", 8, 1024, FP32, "int8", SEED_BASE + 0,
                   protos=("simple",), channels=(1,), chunks=(1 * KiB,),
                   note="8 ranks x 1024 fp32, integers in [-8,8], Simple/1ch/1KiB chunk"),
    # 8 ranks x 4 MiB fp32 uniform [-1, 1); LL vs Simple, channels 1..32.
    "D2": Workload("D2", 8, 1 * MiB, FP32, "uniform", SEED_BASE + 1,
                   protos=("ll", "simple"), channels=(1, 2, 4, 8, 16, 32),
                   note="8 ranks x 4 MiB fp32 uniform[-1,1), LL vs Simple, C in 1..32"),
    # 8 ranks x 32 MiB bf16 normal(0,1), fp32 accumulation; Simple, chunks 128 KiB..2 MiB, C 4..64.
    "D3": Workload("D3", 8, 16 * MiB, BF16, "normal", SEED_BASE + 2,
                   protos=("simple",), channels=(4, 8, 16, 32, 64),
                   chunks=(128 * KiB, 256 * KiB, 512 * KiB, 1 * MiB, 2 * MiB),
                   note="8 ranks x 32 MiB bf16 normal(0,1), fp32 accumulate, Simple"),
    # 8 ranks fp32, 4 KiB..128 MiB in powers of two (the size sweep); count set per size.
    "D4": Workload("D4", 8, 0, FP32, "uniform", SEED_BASE + 3,
                   protos=("ll", "ll128", "simple"), channels=(1, 2, 4, 8, 16, 32, 64),
                   note="8 ranks fp32 uniform[-1,1), 4 KiB..128 MiB, tuned table vs Simple/16",
                   extra={"sizes": tuple(1 << k for k in range(12, 28))}),
    # 8 ranks x 128 MiB fp32 uniform [-1, 1); LL128 vs Simple at 32..64 channels.
    "D5": Workload("D5", 8, 32 * MiB, FP32, "uniform", SEED_BASE + 4,
                   protos=("ll128", "simple"), channels=(32, 48, 64),
                   note="8 ranks x 128 MiB fp32 uniform[-1,1), LL128 vs Simple, C in 32..64"),
}


def sweep_workload(size_bytes: int, dtype: str = FP32, nranks: int = 8) -> Workload:
    """A D4 point: nranks x size_bytes per rank."""
    e = ELEM_BYTES[dtype]
    if size_bytes % e:
        raise ValueError("size must be a multiple of the element size")
    return Workload(f"D4-{size_bytes}", nranks, size_bytes // e, dtype, "uniform",
                    SEED_BASE + 3, note=f"{nranks} ranks x {size_bytes} B {dtype}")
