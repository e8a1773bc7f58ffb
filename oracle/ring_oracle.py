"""CPU oracle for the simulated-ring AllReduce (sum) -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this module.  The HIP library never calls it, and nothing in this
directory shares code, tables or constants with the HIP path.

What is computed
----------------
AllReduce-sum over N rank buffers: every rank ends with
    y[i] = x_0[i] + x_1[i] + ... + x_{N-1}[i]
(paper, section 2, "NCCL and its plugin system": the collective the tuner
steers; section 5.3, Table 2 and Figure 2: the ring AllReduce whose
protocol and channel count the size-aware policy selects).

Floating-point addition is not associative, so the bits depend on the order
in which the ring adds the ranks' contributions.  The paper does not spell
out the ring's data layout (its text defers to NCCL's built-in ring), so
this oracle fixes the following reading of a ring reduce-scatter followed by
an all-gather:

* Segment-major layout.  With A = 16 / (element bytes) elements per 16-byte
  unit, the segment length is seg = roundup(ceil(count / N), A).  Segment s
  covers elements [s*seg, min((s+1)*seg, count)); trailing segments may be
  short or empty.  Channels and chunks subdivide a segment and never change
  which rank starts an element's chain, so the result does not depend on
  protocol, channel count or chunk size.
* The chain for segment s starts at rank s and moves in the ring direction
  r -> r+1:  acc = x_s;  acc = acc + x_{s+1};  ...;  acc = acc + x_{s+N-1}
  (indices mod N), each addition one IEEE binary32 round-to-nearest-even
  operation with subnormals kept.  The last rank of the chain (s-1) owns the
  reduced segment and the all-gather copies it unchanged to every rank.
* bf16 inputs are widened exactly to fp32, the chain runs in fp32, and the
  owner rounds the fp32 sum to bf16 once, round-to-nearest-even, with NaN
  mapped to the quiet NaN 0x7FC0.  Partial sums therefore travel in fp32 and
  only the finished value travels in bf16.

Everything here is plain numpy: a loop over segments and ranks, vectorised
over the elements of one segment.  numpy's float32 ``+`` is elementwise IEEE
RNE, so the loop reproduces the chain bit for bit.
"""
from __future__ import annotations

import numpy as np

F32_UNIT_ROUNDOFF = 2.0 ** -24


def unit_elems(elem_bytes: int) -> int:
    """Elements per 16-byte unit (the alignment of every segment boundary)."""
    if elem_bytes not in (2, 4):
        raise ValueError("element size must be 2 (bf16) or 4 (fp32) bytes")
    return 16 // elem_bytes


def segment_elems(nranks: int, count: int, elem_bytes: int) -> int:
    """seg = roundup(ceil(count / N), A): the length of every full segment."""
    if nranks < 1:
        raise ValueError("nranks must be >= 1")
    a = unit_elems(elem_bytes)
    per_rank = -(-count // nranks)
    return -(-per_rank // a) * a


def _chain_f32(xf32: np.ndarray) -> np.ndarray:
    """Reduce an (N, count) float32 array along the segment-major ring chains."""
    n, count = xf32.shape
    seg = segment_elems(n, count, 4)
    y = np.empty(count, dtype=np.float32)
    if count == 0:
        return y
    for s in range(n):
        lo = s * seg
        hi = min(lo + seg, count)
        if lo >= hi:
            continue
        acc = xf32[s, lo:hi].copy()
        for j in range(1, n):
            acc = acc + xf32[(s + j) % n, lo:hi]
        y[lo:hi] = acc
    return y


def allreduce_f32(x: np.ndarray) -> np.ndarray:
    """fp32 AllReduce-sum of an (N, count) float32 array; returns y (every rank's output)."""
    x = np.asarray(x)
    if x.dtype != np.float32 or x.ndim != 2:
        raise TypeError("expected an (N, count) float32 array")
    return _chain_f32(x)


# --- bf16 -----------------------------------------------------------------
#
# bf16 is the upper half of an IEEE binary32 word.  Widening is exact (append
# sixteen zero bits).  Narrowing rounds to nearest, ties to even, by the
# standard integer method: add 0x7FFF plus the lowest kept bit, then drop the
# low sixteen bits; NaNs become the quiet NaN 0x7FC0.

def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float32 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """float32 values -> uint16 bf16 bit patterns, round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    r[nan] = np.uint16(0x7FC0)
    return r


def allreduce_bf16_acc(xbits: np.ndarray) -> np.ndarray:
    """The fp32 chain sums of bf16 inputs, before the single rounding to bf16."""
    xbits = np.asarray(xbits)
    if xbits.dtype != np.uint16 or xbits.ndim != 2:
        raise TypeError("expected an (N, count) uint16 array of bf16 bits")
    n, count = xbits.shape
    # The segment boundaries are placed on 16-byte units of the bf16 buffer.
    seg = segment_elems(n, count, 2)
    xf = bf16_to_f32(xbits)
    y = np.empty(count, dtype=np.float32)
    for s in range(n):
        lo = s * seg
        hi = min(lo + seg, count)
        if lo >= hi:
            continue
        acc = xf[s, lo:hi].copy()
        for j in range(1, n):
            acc = acc + xf[(s + j) % n, lo:hi]
        y[lo:hi] = acc
    return y


def allreduce_bf16(xbits: np.ndarray) -> np.ndarray:
    """bf16 AllReduce-sum with fp32 accumulation; returns y as uint16 bf16 bits."""
    return f32_to_bf16_rne(allreduce_bf16_acc(xbits))


def allreduce(x: np.ndarray, dtype: str) -> np.ndarray:
    """Dispatch on dtype name: "f32" (float32 array) or "bf16" (uint16 bits)."""
    if dtype == "f32":
        return allreduce_f32(x)
    if dtype == "bf16":
        return allreduce_bf16(x)
    raise ValueError(f"unknown dtype {dtype!r}")


# --- order-free reference and the accuracy bound --------------------------

def sum_f64(x: np.ndarray, dtype: str = "f32") -> np.ndarray:
    """Order-free reference: the rank sum in float64 (exact to ~N * 2^-53)."""
    xf = bf16_to_f32(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)
    return xf.astype(np.float64).sum(axis=0)


def abs_sum_f64(x: np.ndarray, dtype: str = "f32") -> np.ndarray:
    """sum_r |x_r[i]| in float64: the scale of the normwise error bound."""
    xf = bf16_to_f32(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)
    return np.abs(xf.astype(np.float64)).sum(axis=0)


def recursive_sum_gamma(nranks: int) -> float:
    """gamma_{N-1} = (N-1)u / (1 - (N-1)u), u = 2^-24.

    Any order of N-1 binary32 additions satisfies
    |fl(sum) - sum| <= gamma_{N-1} * sum |x_r|  (Higham, recursive summation).
    """
    k = max(nranks - 1, 0)
    return k * F32_UNIT_ROUNDOFF / (1.0 - k * F32_UNIT_ROUNDOFF)


# --- ReduceScatter and AllGather --------------------------------------------
#
# The same ring, run as one half (paper section 2: AllGather is among the
# collectives the tuner steers; section 5.3 measures it).  With `count`
# elements per block and N blocks per full buffer:
#
# * ReduceScatter: rank r receives block r of the sum.  The ring's
#   reduce-scatter ends each block's chain at the rank that keeps it, so
#   block r is summed starting at rank r+1:
#       acc = x_{r+1}[block r]; acc += x_{r+2}[block r]; ...; acc += x_r[block r]
#   (indices mod N), each addition one binary32 RNE operation; bf16 inputs
#   are widened and the result rounded once, as for AllReduce.
# * AllGather: every rank receives [x_0 | x_1 | ... | x_{N-1}]: copies only.

def reduce_scatter_acc(x: np.ndarray, dtype: str) -> np.ndarray:
    """(N, N*count) inputs -> (N, count) fp32 chain sums (before bf16 rounding)."""
    x = np.asarray(x)
    if x.ndim != 2 or x.shape[1] % x.shape[0]:
        raise ValueError("expected an (N, N*count) array")
    n = x.shape[0]
    count = x.shape[1] // n
    xf = bf16_to_f32(x) if dtype == "bf16" else np.asarray(x, np.float32)
    y = np.empty((n, count), np.float32)
    for r in range(n):
        lo, hi = r * count, (r + 1) * count
        start = (r + 1) % n
        acc = xf[start, lo:hi].copy()
        for j in range(1, n):
            acc = acc + xf[(start + j) % n, lo:hi]
        y[r] = acc
    return y


def reduce_scatter(x: np.ndarray, dtype: str) -> np.ndarray:
    """ReduceScatter-sum: (N, N*count) -> (N, count) float32 or uint16 bf16 bits."""
    acc = reduce_scatter_acc(x, dtype)
    return acc if dtype == "f32" else f32_to_bf16_rne(acc).reshape(acc.shape)


def all_gather(x: np.ndarray) -> np.ndarray:
    """AllGather: (N, count) -> every rank's (N*count) concatenation, shape (N*count,)."""
    x = np.asarray(x)
    return x.reshape(-1).copy()
