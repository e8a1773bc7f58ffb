"""Build and call the plain-C oracle (ring_oracle.c) -- TEST INFRASTRUCTURE.

Used by the tests and by the benchmark's CPU-baseline leg.  It computes the
same segment-major ring chains as ring_oracle.py; tests check the two
against each other and against the same pins.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "ring_oracle.c")
LIB = os.path.join(_HERE, "libring_oracle.so")

CFLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC",
          "-std=c11", "-Wall", "-Wextra"]

_lib = None


def build(force: bool = True) -> str:
    """Compile ring_oracle.c into libring_oracle.so next to it."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.run(["gcc", *CFLAGS, SRC, "-o", tmp], check=True)
        os.replace(tmp, LIB)
    return LIB


def lib():
    """Load the C oracle, building it first only if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build(force=True)
        L = ctypes.CDLL(LIB)
        L.ring_oracle_segment.restype = ctypes.c_uint64
        L.ring_oracle_segment.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int]
        for name in ("ring_oracle_f32", "ring_oracle_bf16"):
            f = getattr(L, name)
            f.restype = ctypes.c_int
            f.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_int,
                          ctypes.c_uint64, ctypes.c_int]
        L.ring_oracle_max_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def max_threads() -> int:
    return int(lib().ring_oracle_max_threads())


def segment_elems(nranks: int, count: int, elem_bytes: int) -> int:
    return int(lib().ring_oracle_segment(nranks, count, elem_bytes))


def _ptrs(x: np.ndarray):
    n = x.shape[0]
    arr = (ctypes.c_void_p * max(n, 1))()
    for r in range(n):
        arr[r] = x[r].ctypes.data
    return arr


def allreduce(x: np.ndarray, dtype: str, nthreads: int = 1, out: np.ndarray | None = None) -> np.ndarray:
    """y for an (N, count) float32 ("f32") or uint16 bf16-bits ("bf16") array."""
    x = np.ascontiguousarray(x)
    n, count = x.shape
    if dtype == "f32":
        if x.dtype != np.float32:
            raise TypeError("f32 oracle needs float32 input")
        y = out if out is not None else np.empty(count, np.float32)
        fn = lib().ring_oracle_f32
    elif dtype == "bf16":
        if x.dtype != np.uint16:
            raise TypeError("bf16 oracle needs uint16 bit patterns")
        y = out if out is not None else np.empty(count, np.uint16)
        fn = lib().ring_oracle_bf16
    else:
        raise ValueError(dtype)
    rc = fn(_ptrs(x), y.ctypes.data if count else None, n, count, nthreads)
    if rc != 0:
        raise RuntimeError(f"C oracle failed with {rc}")
    return y
