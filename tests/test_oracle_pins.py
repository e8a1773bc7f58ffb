"""Pins for the CPU oracle: facts fixed by arithmetic, not by the oracle itself.

Each pin is a function of an AllReduce implementation ``impl(x, dtype) -> y``
so that the same pins run against the numpy oracle, the C oracle, and a set
of deliberately broken oracles (planted mistakes) that each pin set must
reject.

Pins:
* all-ones input gives exactly N everywhere (a dropped or repeated hop
  shows as N-1 or N+1);
* integer-valued inputs give the exact integer sum (no rounding occurs);
* hand-worked order-revealing cases fix the chain start and direction per
  segment, in fp32 (tests/golden/order_n4_f32.txt) and in bf16 with fp32
  accumulation (tests/golden/order_n4_bf16.txt, where segments are cut on
  8-element units);
* brute force on tiny order-revealing inputs, fp32 and bf16: every element
  equals the scalar ring chain that starts at its segment's rank, with the
  scalar chain computed by Python doubles rounded to binary32 after every
  add (and, for bf16, rounded once at the end by torch's CPU conversion);
* bf16 rounding cases worked by hand (tests/golden/bf16_single_rounding.txt)
  fix one rounding at the end of an fp32 chain;
* the recursive-summation bound against an order-free float64 sum;
* bf16 round-to-nearest-even against torch's CPU conversion over every
  non-NaN binary32 bit pattern.
"""
from __future__ import annotations

import os
import struct

import numpy as np
import pytest

from oracle import c_oracle
from oracle import ring_oracle as ro

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def numpy_impl(x, dtype):
    return ro.allreduce(x, dtype)


def c_impl(x, dtype):
    return c_oracle.allreduce(x, dtype, nthreads=1)


def c_impl_threads(x, dtype):
    return c_oracle.allreduce(x, dtype, nthreads=4)


IMPLS = {"numpy": numpy_impl, "c": c_impl, "c_omp": c_impl_threads}


def _as_f32(y, dtype):
    return ro.bf16_to_f32(y) if dtype == "bf16" else np.asarray(y, np.float32)


def _ones(n, count, dtype):
    a = np.ones((n, count), np.float32)
    return a if dtype == "f32" else ro.f32_to_bf16_rne(a).reshape(n, count)


# --------------------------------------------------------------------- pins

def pin_all_ones(impl):
    for dtype in ("f32", "bf16"):
        for n in (1, 2, 3, 5, 8, 16):
            for count in (0, 1, 3, 8, 17, 64, 1000, 4099):
                y = _as_f32(impl(_ones(n, count, dtype), dtype), dtype)
                assert y.shape == (count,)
                assert np.all(y == n), (dtype, n, count)


def pin_integer_exact(impl):
    rng = np.random.default_rng(7)
    for dtype in ("f32", "bf16"):
        for n in (2, 3, 4, 8, 16):
            for count in (1, 33, 1000, 5003):
                xi = rng.integers(-8, 9, size=(n, count))
                xf = xi.astype(np.float32)
                x = xf if dtype == "f32" else ro.f32_to_bf16_rne(xf).reshape(n, count)
                y = _as_f32(impl(x, dtype), dtype)
                assert np.array_equal(y.astype(np.int64), xi.sum(axis=0)), (dtype, n, count)


def _read_golden_kv(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if line:
                vals[line[0]] = line[1:]
    return vals


def _torch_bf16_bits(v):
    """float32 values -> bf16 bits by torch's CPU conversion (a library RNE,
    independent of the oracle's own rounding)."""
    import torch

    f = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
    return f.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _read_golden_order(name, dtype):
    vals = _read_golden_kv(name)
    n = int(vals["nranks"][0])
    count = int(vals["count"][0])
    xr = [float(v) for v in vals["x"]]
    y = np.array([float(v) for v in vals["y"]], np.float32)
    x = np.repeat(np.array(xr, np.float32)[:, None], count, axis=1)
    assert x.shape == (n, count)
    if dtype == "bf16":
        xb = _torch_bf16_bits(x).reshape(n, count)
        # every input and every expected value is exact in bf16
        assert np.array_equal(ro.bf16_to_f32(xb), x)
        yb = _torch_bf16_bits(y)
        assert np.array_equal(ro.bf16_to_f32(yb), y)
        return xb, yb
    return x, y.view(np.uint32)


def pin_order_golden(impl):
    x, y = _read_golden_order("order_n4_f32.txt", "f32")
    got = impl(x, "f32")
    assert np.array_equal(got.view(np.uint32), y), got


def pin_order_golden_bf16(impl):
    x, y = _read_golden_order("order_n4_bf16.txt", "bf16")
    got = np.asarray(impl(x, "bf16"))
    assert np.array_equal(got, y), ro.bf16_to_f32(got)


def _f32(v: float) -> float:
    return struct.unpack("<f", struct.pack("<f", v))[0]


def _scalar_chain(vals, start):
    n = len(vals)
    acc = _f32(vals[start])
    for j in range(1, n):
        # Both operands are binary32 values of moderate range, so the double
        # sum is exact and packing it rounds once, to nearest even.
        acc = _f32(acc + vals[(start + j) % n])
    return acc


ORDER_VALUES = np.array([2.0 ** 24, -(2.0 ** 24), 2.0 ** 25, 1.0, -1.0, 3.0, 0.5, 2.0], np.float32)


def pin_brute_force_rotations(impl):
    rng = np.random.default_rng(11)
    informative = 0
    for n in (2, 3, 4, 5, 8):
        for count in (1, 5, 8, 13, 32, 64):
            x = rng.choice(ORDER_VALUES, size=(n, count)).astype(np.float32)
            got = impl(x, "f32")
            a = 4
            seg = -(-(-(-count // n)) // a) * a
            for i in range(count):
                vals = [float(x[r, i]) for r in range(n)]
                chains = [_scalar_chain(vals, s) for s in range(n)]
                want = chains[i // seg]
                assert float(got[i]) == want, (n, count, i, vals, chains, float(got[i]))
                if any(c != want for c in chains):
                    informative += 1
    assert informative > 100  # the inputs really do tell chain orders apart


def pin_brute_force_rotations_bf16(impl):
    """bf16 inputs (every order value is exact in bf16), fp32 chains, one
    rounding at the end; segments are cut on 16-byte units of the bf16
    buffer, A = 8 elements.  The counts put segment boundaries where the
    fp32 unit (A = 4) would cut them differently."""
    rng = np.random.default_rng(12)
    informative = 0
    for n in (2, 3, 4, 5, 8):
        for count in (1, 5, 13, 32, 64, 100, 250, 333):
            xf = rng.choice(ORDER_VALUES, size=(n, count)).astype(np.float32)
            xb = _torch_bf16_bits(xf).reshape(n, count)
            assert np.array_equal(ro.bf16_to_f32(xb), xf)
            got = np.asarray(impl(xb, "bf16"))
            a = 8
            seg = -(-(-(-count // n)) // a) * a
            for i in range(count):
                vals = [float(xf[r, i]) for r in range(n)]
                chains = [_scalar_chain(vals, s) for s in range(n)]
                rounded = [int(_torch_bf16_bits(np.array([c], np.float32))[0]) for c in chains]
                want = rounded[i // seg]
                assert int(got[i]) == want, (n, count, i, vals, chains, hex(int(got[i])))
                if any(c != want for c in rounded):
                    informative += 1
    assert informative > 100  # chain orders stay distinguishable after rounding


def _read_golden_bf16():
    cases = []
    with open(os.path.join(GOLDEN, "bf16_single_rounding.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line.startswith("case"):
                continue
            name, vals, want = [p.strip() for p in line[4:].split("|")]
            cases.append((name, [float(v) for v in vals.split()], float(want)))
    return cases


def pin_bf16_single_rounding(impl):
    cases = _read_golden_bf16()
    assert len(cases) >= 5
    for name, vals, want in cases:
        n = len(vals)
        xf = np.repeat(np.array(vals, np.float32)[:, None], 8, axis=1)
        xb = ro.f32_to_bf16_rne(xf).reshape(n, 8)
        # the inputs themselves must be exact bf16 values
        assert np.array_equal(ro.bf16_to_f32(xb), xf), name
        y = ro.bf16_to_f32(impl(xb, "bf16"))
        assert np.all(y == np.float32(want)), (name, y, want)


def pin_fp64_bound(impl):
    rng = np.random.default_rng(3)
    for n in (2, 8, 16):
        x = (rng.random((n, 20011), dtype=np.float32) * 2 - 1).astype(np.float32)
        y = impl(x, "f32").astype(np.float64)
        s = ro.sum_f64(x)
        scale = ro.abs_sum_f64(x)
        err = np.abs(y - s)
        assert np.all(err <= ro.recursive_sum_gamma(n) * scale)
        assert np.all(err <= 1e-5 * scale)
    # bf16: the fp32 accumulator obeys the same bound; the rounded output is
    # within one bf16 unit in the last place of the exact sum.
    xb = ro.f32_to_bf16_rne(rng.standard_normal((8, 20011), dtype=np.float32)).reshape(8, 20011)
    s = ro.sum_f64(xb, "bf16")
    yb = ro.bf16_to_f32(impl(xb, "bf16")).astype(np.float64)
    ulp = np.maximum(np.abs(s), 2.0 ** -126) * 2.0 ** -7
    assert np.all(np.abs(yb - s) <= ulp + ro.recursive_sum_gamma(8) * ro.abs_sum_f64(xb, "bf16"))


PINS = [pin_all_ones, pin_integer_exact, pin_order_golden, pin_order_golden_bf16, pin_brute_force_rotations,
        pin_brute_force_rotations_bf16, pin_bf16_single_rounding, pin_fp64_bound]


@pytest.mark.parametrize("impl_name", sorted(IMPLS))
@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin, impl_name):
    pin(IMPLS[impl_name])


# ------------------------------------------------------- planted mistakes
#
# Each mutant is a plausible wrong oracle.  The pin set must reject every one
# of them; otherwise the pins would not be worth trusting.

def _mutant(chain_start, order="fwd", drop_last=False, per_hop_bf16=False, no_roundup=False,
            negate=False, bf16_unit=None, bf16_start=None):
    """bf16_unit / bf16_start: mistakes confined to the bf16 path (segments
    cut on a unit of bf16_unit elements; chains started by bf16_start)."""
    def impl(x, dtype):
        n, count = x.shape
        e = 4 if dtype == "f32" else 2
        a = 16 // e
        if dtype == "bf16" and bf16_unit is not None:
            a = bf16_unit
        per = -(-count // n)
        seg = per if no_roundup else -(-per // a) * a
        xf = ro.bf16_to_f32(x) if dtype == "bf16" else x
        y = np.empty(count, np.float32)
        if count == 0:
            return y if dtype == "f32" else ro.f32_to_bf16_rne(y)
        start_of = bf16_start if (dtype == "bf16" and bf16_start is not None) else chain_start
        for s in range(n):
            lo, hi = s * seg, min((s + 1) * seg, count)
            if lo >= hi:
                continue
            st = start_of(s, n)
            acc = xf[st, lo:hi].copy()
            terms = range(1, n - 1) if drop_last else range(1, n)
            for j in terms:
                r = (st + j) % n if order == "fwd" else (st - j) % n
                t = xf[r, lo:hi]
                acc = acc - t if (negate and j == 1) else acc + t
                if per_hop_bf16 and dtype == "bf16":
                    acc = ro.bf16_to_f32(ro.f32_to_bf16_rne(acc))
            y[lo:hi] = acc
        return y if dtype == "f32" else ro.f32_to_bf16_rne(y)
    return impl


MUTANTS = {
    "start_next_rank": _mutant(lambda s, n: (s + 1) % n),
    "start_rank0": _mutant(lambda s, n: 0),
    "reverse_direction": _mutant(lambda s, n: s, order="rev"),
    "drop_last_term": _mutant(lambda s, n: s, drop_last=True),
    "per_hop_bf16": _mutant(lambda s, n: s, per_hop_bf16=True),
    "no_segment_roundup": _mutant(lambda s, n: s, no_roundup=True),
    "wrong_sign": _mutant(lambda s, n: s, negate=True),
    # mistakes only the bf16 path makes
    "bf16_fp32_unit": _mutant(lambda s, n: s, bf16_unit=4),
    "bf16_start_next_rank": _mutant(lambda s, n: s, bf16_start=lambda s, n: (s + 1) % n),
    "bf16_start_rank0": _mutant(lambda s, n: s, bf16_start=lambda s, n: 0),
}


def test_unmutated_reference_passes():
    good = _mutant(lambda s, n: s)
    for pin in PINS:
        pin(good)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name):
    impl = MUTANTS[name]
    failed = []
    for pin in PINS:
        try:
            pin(impl)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"no pin rejects mutant {name}"


# --------------------------------------------------------------- geometry

def test_segment_rule_examples():
    # seg = roundup(ceil(count / N), 16 / e)
    assert ro.segment_elems(8, 1024, 4) == 128
    assert ro.segment_elems(8, 1, 4) == 4
    assert ro.segment_elems(8, 33, 4) == 8
    assert ro.segment_elems(8, 16 * 1024 * 1024, 2) == 2 * 1024 * 1024
    assert ro.segment_elems(3, 8, 2) == 8
    assert ro.segment_elems(1, 5, 4) == 8
    for n in (1, 2, 3, 7, 8, 16):
        for count in (0, 1, 2, 15, 16, 17, 1000, 12345):
            for e in (2, 4):
                assert ro.segment_elems(n, count, e) == c_oracle.segment_elems(n, count, e)


def test_c_oracle_matches_numpy_oracle_bits():
    rng = np.random.default_rng(5)
    for dtype in ("f32", "bf16"):
        for n in (1, 2, 3, 8, 16):
            for count in (0, 1, 7, 100, 4096, 65537):
                xf = rng.standard_normal((n, count), dtype=np.float32)
                x = xf if dtype == "f32" else ro.f32_to_bf16_rne(xf).reshape(n, count)
                a = ro.allreduce(x, dtype)
                for t in (1, 3):
                    b = c_oracle.allreduce(x, dtype, nthreads=t)
                    assert a.tobytes() == b.tobytes(), (dtype, n, count, t)


def test_subnormals_kept():
    # 2^-149 + 2^-149 = 2^-148: a flush-to-zero implementation would give 0.
    tiny = np.float32(2.0 ** -149)
    x = np.full((2, 4), tiny, np.float32)
    for impl in IMPLS.values():
        y = impl(x, "f32")
        assert np.all(y == np.float32(2.0 ** -148))
    # x + (-x) = +0
    x = np.array([[1.5] * 4, [-1.5] * 4], np.float32)
    for impl in IMPLS.values():
        y = impl(x, "f32")
        assert np.all(y.view(np.uint32) == 0)


# ------------------------------------------------------------ bf16 rounding

def test_bf16_rne_hand_cases():
    cases = {
        0x3F800000: 0x3F80,  # 1.0
        0x3F808000: 0x3F80,  # 1 + 2^-8: tie, even stays
        0x3F818000: 0x3F82,  # 1 + 3*2^-8: tie, odd rounds up
        0x3F808001: 0x3F81,  # just above the tie
        0x7F7FFFFF: 0x7F80,  # max float rounds up to +inf
        0xFF800000: 0xFF80,  # -inf stays
        0x00000001: 0x0000,  # smallest subnormal rounds to +0
        0x80000000: 0x8000,  # -0
        0x7FC00000: 0x7FC0,  # quiet NaN
        0x7F800001: 0x7FC0,  # signalling NaN -> quiet NaN
        0xFFFFFFFF: 0x7FC0,
    }
    u = np.array(list(cases), np.uint32)
    got = ro.f32_to_bf16_rne(u.view(np.float32))
    assert [int(v) for v in got] == list(cases.values())


def test_bf16_rne_stratified_vs_torch():
    """Every upper half-word with the lower half-words that decide rounding.

    Rounding to bf16 depends only on the kept upper 16 bits (their lowest bit
    breaks ties) and on where the dropped lower 16 bits sit relative to the
    half-way point 0x8000, so every upper half combined with lower halves
    around 0, 0x8000 and 0xFFFF, plus random ones, covers each case.
    """
    import torch

    lows = np.array([0x0000, 0x0001, 0x0002, 0x3FFF, 0x7FFE, 0x7FFF, 0x8000, 0x8001, 0x8002,
                     0xBFFF, 0xFFFE, 0xFFFF], np.uint32)
    rng = np.random.default_rng(1)
    lows = np.concatenate([lows, rng.integers(0, 1 << 16, 20, dtype=np.uint32)])
    u = ((np.arange(1 << 16, dtype=np.uint32)[:, None] << np.uint32(16)) | lows[None, :]).ravel()
    f = u.view(np.float32)
    ours = ro.f32_to_bf16_rne(f)
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(f)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.all(ours[nan] == 0x7FC0)


def _rne_chunk_mismatches(start: int, step: int) -> int:
    """Bit patterns in [start, start + step) where the oracle's RNE differs
    from torch's CPU bf16 conversion (NaNs: the oracle's canonical 0x7FC0)."""
    import torch

    torch.set_num_threads(1)
    u = np.arange(step, dtype=np.uint32) + np.uint32(start)
    f = u.view(np.float32)
    ours = ro.f32_to_bf16_rne(f)
    ref = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(f)
    return int(np.count_nonzero(ours[~nan] != ref[~nan]) + np.count_nonzero(ours[nan] != 0x7FC0))


def test_bf16_rne_exhaustive_vs_torch():
    """Every binary32 bit pattern: oracle RNE == torch CPU bf16 conversion,
    in 256 blocks spread over worker processes."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor

    step = 1 << 24
    starts = list(range(0, 1 << 32, step))
    workers = max(1, min(8, os.cpu_count() or 1))
    with ProcessPoolExecutor(workers, mp_context=mp.get_context("spawn")) as pool:
        bad = list(pool.map(_rne_chunk_mismatches, starts, [step] * len(starts)))
    assert sum(bad) == 0, [hex(s) for s, b in zip(starts, bad) if b]


# ------------------------------------------------ ReduceScatter / AllGather
#
# Pins of the ReduceScatter oracle, as functions of an implementation
# ``rs(x, dtype) -> (N, count)`` (float32 values or uint16 bf16 bits), run on
# the oracle and on planted mistakes as above.

def rs_pin_golden(rs):
    for name, dtype in (("reduce_scatter_order_n4_f32.txt", "f32"), ("reduce_scatter_order_n4_bf16.txt", "bf16")):
        vals = _read_golden_kv(name)
        n, count = int(vals["nranks"][0]), int(vals["count"][0])
        x = np.repeat(np.array([float(v) for v in vals["x"]], np.float32)[:, None], n * count, axis=1)
        if dtype == "bf16":
            xb = _torch_bf16_bits(x).reshape(n, n * count)
            assert np.array_equal(ro.bf16_to_f32(xb), x)
            x = xb
        y = _as_f32(np.asarray(rs(x, dtype)).reshape(-1), dtype).reshape(n, count)
        for r, want in enumerate(vals["y"]):
            assert np.all(y[r] == np.float32(float(want))), (name, r, y[r])


def rs_pin_invariants(rs):
    rng = np.random.default_rng(21)
    for dtype in ("f32", "bf16"):
        for n in (1, 2, 3, 8, 16):
            for count in (8, 104):
                # all ones -> n
                ones = np.ones((n, n * count), np.float32)
                xo = ones if dtype == "f32" else ro.f32_to_bf16_rne(ones).reshape(n, n * count)
                y = _as_f32(np.asarray(rs(xo, dtype)).reshape(-1), dtype)
                assert np.all(y == n)
                # integers exact; block r of the sum lands on rank r
                xi = rng.integers(-8, 9, size=(n, n * count))
                xf = xi.astype(np.float32)
                x = xf if dtype == "f32" else ro.f32_to_bf16_rne(xf).reshape(n, n * count)
                y = _as_f32(np.asarray(rs(x, dtype)).reshape(-1), dtype).reshape(n, count)
                want = xi.sum(axis=0).reshape(n, count)
                assert np.array_equal(y.astype(np.int64), want)


def rs_pin_brute_force_chain(rs):
    """Every element of block r equals the scalar chain that starts at rank
    r+1 (fp32), or that chain rounded once by torch's conversion (bf16)."""
    rng = np.random.default_rng(22)
    informative = {"f32": 0, "bf16": 0}
    for dtype in ("f32", "bf16"):
        for n in (2, 3, 5, 8):
            count = 64
            xf = rng.choice(ORDER_VALUES, size=(n, n * count)).astype(np.float32)
            x = xf if dtype == "f32" else _torch_bf16_bits(xf).reshape(n, n * count)
            y = np.asarray(rs(x, dtype)).reshape(n, count)
            for r in range(n):
                for i in range(count):
                    vals = [float(xf[q, r * count + i]) for q in range(n)]
                    chains = [_scalar_chain(vals, s) for s in range(n)]
                    if dtype == "f32":
                        cand = [np.float32(c).view(np.uint32) for c in chains]
                        got = np.float32(y[r, i]).view(np.uint32)
                    else:
                        cand = [int(_torch_bf16_bits(np.array([c], np.float32))[0]) for c in chains]
                        got = int(y[r, i])
                    want = cand[(r + 1) % n]
                    assert got == want, (dtype, n, r, i, vals, chains)
                    if any(c != want for c in cand):
                        informative[dtype] += 1
    assert min(informative.values()) > 50, informative


RS_PINS = [rs_pin_golden, rs_pin_invariants, rs_pin_brute_force_chain]


def test_reduce_scatter_pins_hold_for_the_oracle():
    for pin in RS_PINS:
        pin(ro.reduce_scatter)


def _rs_mutant(start_shift=1, reverse=False, bf16_only=False, per_hop_bf16=False):
    """A ReduceScatter oracle with one planted mistake: block r's chain starts
    at rank r + start_shift, or runs against the ring direction, or rounds
    to bf16 after every hop; bf16_only confines the mistake to bf16."""
    def rs(x, dtype):
        n = x.shape[0]
        count = x.shape[1] // n
        xf = ro.bf16_to_f32(x) if dtype == "bf16" else np.asarray(x, np.float32)
        wrong = dtype == "bf16" or not bf16_only
        y = np.empty((n, count), np.float32)
        for r in range(n):
            lo, hi = r * count, (r + 1) * count
            st = (r + (start_shift if wrong else 1)) % n
            acc = xf[st, lo:hi].copy()
            for j in range(1, n):
                q = (st - j) % n if (wrong and reverse) else (st + j) % n
                acc = acc + xf[q, lo:hi]
                if wrong and per_hop_bf16 and dtype == "bf16":
                    acc = ro.bf16_to_f32(ro.f32_to_bf16_rne(acc)).reshape(acc.shape)
            y[r] = acc
        return y if dtype == "f32" else ro.f32_to_bf16_rne(y).reshape(n, count)
    return rs


RS_MUTANTS = {
    "start_at_owner": _rs_mutant(start_shift=0),
    "bf16_start_at_owner": _rs_mutant(start_shift=0, bf16_only=True),
    "bf16_start_two_late": _rs_mutant(start_shift=2, bf16_only=True),
    "bf16_reverse_direction": _rs_mutant(reverse=True, bf16_only=True),
    "bf16_per_hop_rounding": _rs_mutant(per_hop_bf16=True, bf16_only=True),
}


def test_reduce_scatter_unmutated_passes():
    for pin in RS_PINS:
        pin(_rs_mutant())


@pytest.mark.parametrize("name", sorted(RS_MUTANTS))
def test_reduce_scatter_pins_reject_mutant(name):
    failed = []
    for pin in RS_PINS:
        try:
            pin(RS_MUTANTS[name])
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"no ReduceScatter pin rejects mutant {name}"


def test_all_gather_is_concatenation():
    x = np.arange(24, dtype=np.float32).reshape(4, 6)
    assert np.array_equal(ro.all_gather(x), np.arange(24, dtype=np.float32))
