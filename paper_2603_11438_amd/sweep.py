"""Measure {protocol, channels, chunk, waves} per message size and derive the
size -> decision table compiled into libar (csrc/tuner_table.inc).

This is how the paper's size-aware policy is obtained (section 5.3: a sweep
of the ring's choices per message size, then a per-size selection), redone
on MI355X for the simulated ring.

    python -m paper_2603_11438_amd.sweep measure --out sweep.jsonl
    python -m paper_2603_11438_amd.sweep table sweep.jsonl --emit csrc/tuner_table.inc
    python -m paper_2603_11438_amd.sweep validate --out validate.jsonl
    python -m paper_2603_11438_amd.sweep stability --coll allgather --out stability.jsonl
    python -m paper_2603_11438_amd.sweep latency --out latency.jsonl
    python -m paper_2603_11438_amd.sweep configs --out configs.jsonl
    python -m paper_2603_11438_amd.sweep trace --out trace.jsonl

`measure` times each candidate as the device runs it (calls captured in a
HIP graph and replayed), so small messages are ranked by kernel time rather
than by the host's launch rate; `validate` times end-to-end calls launched
from the host, as an application sees them (`--timing` switches either).
Every timing loop runs out of place on fixed inputs through a bound call
(one C call per run); `--dtype bf16` sweeps or validates bf16 data, which
has an AllReduce table of its own.

Selection rule per size, for the ring's columns: the highest median bus
bandwidth wins; candidates within 2 % of the best count as ties and are
broken by fewer channels, then fewer wire bytes (Simple < LL128 < LL), then
smaller chunk, then the higher bandwidth, channels and chunk counted as the
plan resolved them; when the fixed default is within 2 % the row defers to
it.  The direct algorithm's columns take its fastest {workgroups per
segment, waves, units per thread}, ties within 2 % going to fewer resolved
workgroups.  The algorithm column picks the faster of the two (the direct
algorithm on a tie: it moves fewer bytes).
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import paper_2603_11438_amd as ar

SIZES = [1 << k for k in range(12, 28)]
DEFAULT_CHUNK = 256 << 10   # the library's Simple chunk when no tuner opinion
DEFAULT_WAVES = 4
WIRE_RANK = {"simple": 0, "ll128": 1, "ll": 2}
CHUNKS = {"ll": (4096, 16384, 65536), "ll128": (15360, 61440, 245760),
          "simple": (16384, 65536, 262144, 1048576)}


def _uniform(count, dtype, gen):
    """count values uniform in [-1, 1) in the data type (bf16: rounded)."""
    import torch

    t = torch.rand(count, device="cuda:0", generator=gen) * 2 - 1
    return t if dtype == "f32" else t.to(torch.bfloat16)


def _runner(plan, ts):
    """A call of the plan out of place: the inputs ts (each rank's full
    buffer) stay fixed and the results go to separate buffers.  Timing loops
    use it because repeated in-place AllReduces feed each call the previous
    call's sums, which grow about N-fold per call and are inf or NaN within
    a few dozen calls, and the HBM rate depends on the values moved."""
    import torch

    coll, count = plan.info["coll"], plan.info["count"]
    if coll == ar.AR_COLL_ALLGATHER:
        send = [t[:count] for t in ts]
        recv = [torch.empty_like(t) for t in ts]
    elif coll == ar.AR_COLL_REDUCESCATTER:
        send = ts
        recv = [torch.empty(count, dtype=t.dtype, device=t.device) for t in ts]
    else:
        send = ts
        recv = [torch.empty_like(t) for t in ts]
    # one bound call per stream: the buffers are checked once, and a call
    # costs the library's launch, not the binding's per-call checks
    bound = {}

    def run(stream):
        key = None if stream is None else stream.cuda_stream
        fn = bound.get(key)
        if fn is None:
            fn = bound[key] = plan.bind(send, recv, stream)
        fn()

    return run


def _timer(plan, ts, stream, min_total_s=2e-3, reps=5, warm=3, graph=False):
    """Seconds per call, `reps` samples, out of place on fixed inputs.
    Eager: k calls launched back to back from the host (small messages then
    measure the host's launch rate).  Graph: k calls captured in one HIP
    graph and replayed, which measures the device's time per call."""
    import torch

    run = _runner(plan, ts)
    for _ in range(warm):
        run(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(stream)
    torch.cuda.synchronize()
    one = max(time.perf_counter() - t0, 1e-6)
    k = max(10, min(2000, int(min_total_s / one)))
    if graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for _ in range(k):
                run(side)
        g.replay()
        torch.cuda.synchronize()
        out = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            e1.synchronize()
            out.append(e0.elapsed_time(e1) / k / 1e3)
        del g
        if plan.status() != ar.AR_OK:
            raise RuntimeError("timeout during sweep")
        return out
    out = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(k):
            run(stream)
        e1.record(stream)
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) / k / 1e3)
    if plan.status() != ar.AR_OK:
        raise RuntimeError("timeout during sweep")
    return out


DIRECT_PARTS = (0, 16, 32, 64, 96, 128, 256)
DIRECT_WAVES = (1, 2, 4, 8, 16)
DIRECT_UNROLL = (1, 2)


def grid(size, protos=("ll", "ll128", "simple"), channels=(1, 2, 4, 8, 16, 32, 64), waves=(2, 4, 8),
         chunks=None):
    for parts in DIRECT_PARTS:
        for w in DIRECT_WAVES:
            for u in DIRECT_UNROLL:
                yield dict(algo="direct", nchannels=parts, nwaves=w, direct_unroll=u)
    chunks = chunks or CHUNKS
    for p in protos:
        for c in channels:
            for w in waves:
                for k in chunks[p]:
                    # chunks far beyond a channel's share repeat the same geometry
                    if k > 4 * max(size // 8 // c, 16) and k != chunks[p][0]:
                        continue
                    yield dict(proto=p, nchannels=c, nwaves=w, chunk_bytes=k)


def bus_bw(coll, size, seconds, n):
    """Bus bandwidth, GB/s: AllReduce S/t * 2(N-1)/N; ReduceScatter and
    AllGather S/t * (N-1)/N, with S the bytes of each rank's full buffer."""
    factor = 2.0 if coll == "allreduce" else 1.0
    return size / seconds * factor * (n - 1) / n / 1e9


# A reduced ring grid for ReduceScatter / AllGather sweeps.
SMALL_GRID = dict(channels=(4, 16, 32, 64), waves=(4, 8),
                  chunks={"ll": (4096, 16384), "ll128": (15360, 61440), "simple": (65536, 262144)})


def measure(args):
    import torch

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    sizes = [int(s) for s in args.sizes.split(",")] if args.sizes else SIZES
    n, coll, dtype = args.nranks, args.coll, args.dtype
    e = 4 if dtype == "f32" else 2
    with open(args.out, "a") as fo:
        for size in sizes:
            count = size // e if coll == "allreduce" else size // e // n
            if count == 0:
                continue
            g = torch.Generator(device="cuda:0").manual_seed(11438)
            ts = [_uniform(size // e, dtype, g) for _ in range(n)]
            for cfg in grid(size, **({} if coll == "allreduce" else SMALL_GRID)):
                if args.algo and cfg.get("algo", "ring") != args.algo:
                    continue
                try:
                    plan = ar.Plan(n, count, dtype, coll=coll, **cfg)
                except ar.ARError as e:
                    continue
                times = _timer(plan, ts, stream, graph=args.timing == "graph")
                info = plan.info
                med = statistics.median(times)
                rec = {"coll": coll, "dtype": dtype, "timing": args.timing, "size": size, "nranks": n, "proto": info["proto_name"], "chunk_bytes": 0, **cfg,
                       "algo": info["algo_name"], "parts_eff": info["nchannels"],
                       "chunk_eff": info["chunk_elems"] * (4 if dtype == "f32" else 2),
                       "t_med_us": med * 1e6, "t_min_us": min(times) * 1e6, "t_max_us": max(times) * 1e6,
                       "busbw": bus_bw(coll, size, med, n)}
                fo.write(json.dumps(rec) + "\n")
                plan.destroy()
            fo.flush()
            print(f"sweep: size {size} done", flush=True)
            del ts
            torch.cuda.empty_cache()


def default_row(size, rs, nranks=8, coll="allreduce", dtype="f32"):
    """The measured row that has the fixed default's geometry (Simple, 16
    channels, default chunk and waves), if the sweep contains it."""
    e = 4 if dtype == "f32" else 2
    count = size // e if coll == "allreduce" else size // e // nranks
    g = ar.ar_plan_geometry(ar.make_desc(nranks, count, dtype, "simple", 16, DEFAULT_CHUNK,
                                         nwaves=DEFAULT_WAVES, coll=coll))
    for r in rs:
        if (r["proto"], r["nchannels"], r["nwaves"]) == ("simple", 16, DEFAULT_WAVES) and \
                r["chunk_eff"] == g["chunk_elems"] * e:
            return r
    return None


def select(rows, tie=0.02, coll="allreduce", dtype="f32", validated=None):
    """Per size: {"ring": ring choice, "direct": direct choice or None, "algo": "ring" | "direct"}.

    validated: {size: ring/default bus-bandwidth ratio measured by `validate`
    on fresh repeats}.  A ring choice whose validated ratio is below 1 + tie
    defers to the fixed default after all: the selection is made on one set
    of repeats and must hold on another."""
    ring = select_ring([r for r in rows if r.get("algo", "ring") == "ring"], tie, coll, dtype)
    for size, rr in ring.items():
        ratio = (validated or {}).get(size)
        if ratio is not None and rr["proto"] != "default" and ratio < 1 + tie:
            ring[size] = dict(rr, proto="default", validated_ratio=ratio)
    out = {}
    for size, rr in ring.items():
        ds = [r for r in rows if r["size"] == size and r.get("algo") == "direct"]
        d = None
        if ds:
            best = max(r["busbw"] for r in ds)
            ties = [r for r in ds if r["busbw"] >= (1 - tie) * best]
            # parts_eff: a row asking for the size rule (0) competes with the
            # part count that rule resolved to
            ties.sort(key=lambda r: (r.get("parts_eff", r["nchannels"]), -r["busbw"]))
            d = ties[0]
        algo = "direct" if d is not None and d["busbw"] >= (1 - tie) * rr["busbw"] else "ring"
        out[size] = {"ring": rr, "direct": d, "algo": algo}
    return out


def select_ring(rows, tie=0.02, coll="allreduce", dtype="f32"):
    """Per size: the highest median bus bandwidth; candidates within `tie` of
    the best are ties, broken by fewer channels, fewer wire bytes, smaller
    chunk, then the higher bandwidth.  When the fixed default is itself within `tie` of the
    best, the row defers to it (the paper's policy also leaves sizes where
    its choice does not help to the library default)."""
    by = {}
    for r in rows:
        by.setdefault(r["size"], []).append(r)
    table = {}
    for size, rs in sorted(by.items()):
        best = max(r["busbw"] for r in rs)
        dflt = default_row(size, rs, coll=coll, dtype=dtype)
        if dflt is not None and dflt["busbw"] >= (1 - tie) * best:
            table[size] = dict(dflt, proto="default")
            continue
        ties = [r for r in rs if r["busbw"] >= (1 - tie) * best]
        ties.sort(key=lambda r: (r.get("parts_eff", r["nchannels"]), WIRE_RANK[r["proto"]],
                                 r.get("chunk_eff", r["chunk_bytes"]), -r["busbw"]))
        table[size] = ties[0]
    return table


TABLE_NAMES = {("allreduce", "f32"): "kTableAllReduce", ("allreduce", "bf16"): "kTableAllReduceBf16",
               ("reducescatter", "f32"): "kTableReduceScatter", ("reducescatter", "bf16"): "kTableReduceScatterBf16",
               ("allgather", "f32"): "kTableAllGather", ("allgather", "bf16"): "kTableAllGatherBf16"}


def emit(tables, path):
    """tables: {(coll, dtype): per-size selection}; writes one C array per
    collective and data type (a bf16 table repeats the fp32 rows when no
    bf16 sweep is given)."""
    out = []
    for key in TABLE_NAMES:
        table = tables.get(key)
        src = key
        if table is None and key[1] != "f32":
            src = (key[0], "f32")
            table = tables.get(src, {})
        out.append(emit_one(table or {}, key, measured_as=src))
    with open(path, "w") as f:
        f.write("\n".join(out))


def emit_one(table, key, measured_as=None):
    coll, dtype = key
    measured_as = measured_as or key
    names = {"ll": "AR_PROTO_LL", "ll128": "AR_PROTO_LL128", "simple": "AR_PROTO_SIMPLE",
             "default": "AR_PROTO_AUTO"}
    lines = [
        f"// {coll}, {dtype}: MI355X size -> {{algorithm; ring protocol, channels, chunk, waves;",
        f"// direct workgroups per segment, waves, units per thread}} table for 8-rank {measured_as[1]}",
        "// collectives, one row per power-of-two size of each rank's full buffer from",
        "// 4 KiB to 128 MiB.  A message of S bytes uses the row of the smallest size",
        "// >= S (sizes below 4 KiB use the first row, above 128 MiB the last).",
        "//",
        "// Same form as the paper's size-aware policy (section 5.3: one protocol for",
        "// the middle sizes, another for the large sizes); the values were measured",
        "// on MI355X by paper_2603_11438_amd/sweep.py (highest median bus bandwidth,",
        "// ties within 2% broken by fewer channels, fewer wire bytes, smaller chunk).",
        "// AR_PROTO_AUTO ring columns defer to the fixed default (Simple, 16 channels):",
        "// there the default measured within 2% of the best ring choice (on the",
        "// sweep, or when validated on fresh repeats).  The",
        "// algorithm column picks the faster of the best ring and the best direct",
        "// choice (direct on a tie, as it moves fewer bytes).",
        "//",
        "// columns: log2(size), ring proto, nchannels, chunk_bytes, nwaves, algorithm,",
        "//          direct parts, direct waves, direct unroll   [busBW GB/s: ring / direct]",
        f"static const TableRow {TABLE_NAMES[key]}[] = {{",
    ]
    if not table:
        lines.append("    {27, AR_PROTO_AUTO, 0, 0, 0, AR_ALGO_AUTO, 0, 0, 0},  // not measured: defer to the default")
    for size, row in sorted(table.items()):
        lg = size.bit_length() - 1
        r, d = row["ring"], row["direct"]
        ring_cols = ("AR_PROTO_AUTO, 0, 0, 0" if r["proto"] == "default" else
                     f"{names[r['proto']]}, {r['nchannels']}, {r['chunk_bytes']}, {r['nwaves']}")
        algo = "AR_ALGO_DIRECT" if row["algo"] == "direct" else "AR_ALGO_RING"
        dcols = f"{d['nchannels']}, {d['nwaves']}, {d.get('direct_unroll', 0)}" if d else "0, 0, 0"
        dbw = f"{d['busbw']:.1f}" if d else "-"
        note = " (ring validated within 2 % of the default: defers)" if "validated_ratio" in r else ""
        lines.append(f"    {{{lg}, {ring_cols}, {algo}, {dcols}}},  // {r['busbw']:.1f} / {dbw}{note}")
    lines.append("};")
    return "\n".join(lines) + "\n"


def table_cmd(args):
    rows = []
    for f in args.jsonl:
        rows += [json.loads(l) for l in open(f) if l.strip()]
    val = {}
    for f in getattr(args, "validated", None) or []:
        for l in open(f):
            if l.strip():
                v = json.loads(l)
                val.setdefault((v.get("coll", "allreduce"), v.get("dtype", "f32")), {})[v["size"]] = v["ratio_ring"]
    tables = {}
    for coll, dtype in TABLE_NAMES:
        rs = [r for r in rows if r.get("coll", "allreduce") == coll and r.get("dtype", "f32") == dtype]
        if rs:
            tables[(coll, dtype)] = select(rs, coll=coll, dtype=dtype, validated=val.get((coll, dtype)))
    for (coll, dtype), table in tables.items():
        print(f"== {coll} {dtype}")
        print_table(table)
    if args.emit:
        emit(tables, args.emit)


def print_table(table):
    for size, row in sorted(table.items()):
        r, d = row["ring"], row["direct"]
        ds = (f"direct P={d['nchannels']:3} W={d['nwaves']:2} U={d.get('direct_unroll', 0)} busBW={d['busbw']:7.1f}"
              if d else "direct -")
        print(f"{size:>10} {row['algo']:6} | ring {r['proto']:7} C={r['nchannels']:3} chunk={r['chunk_bytes']:8} "
              f"W={r['nwaves']} busBW={r['busbw']:6.1f} | {ds}")


def validate(args):
    """Tuned table (ar_plan with AUTO) vs the fixed Simple/16 default, fresh repeats."""
    import torch

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    n, coll, dtype = args.nranks, args.coll, args.dtype
    e = 4 if dtype == "f32" else 2
    sizes = [int(s) for s in args.sizes.split(",")] if args.sizes else SIZES
    with open(args.out, "a") as fo:
        for size in sizes:
            count = size // e if coll == "allreduce" else size // e // n
            if count == 0:
                continue
            g = torch.Generator(device="cuda:0").manual_seed(11438 + 100)
            ts = [_uniform(size // e, dtype, g) for _ in range(n)]
            res = {}
            bad = lambda ctx: {"proto": ar.AR_PROTO_SIMPLE, "nchannels": 1, "algo": ar.AR_ALGO_RING}
            for name, tuner, algo in (("tuned", None, "auto"), ("tuned_ring", None, "ring"),
                                      ("default", "fixed_default", "auto"), ("bad_channels", bad, "auto")):
                ar.ar_set_tuner(tuner)
                plan = ar.Plan(n, count, dtype, proto="auto", algo=algo, coll=coll)
                ar.ar_set_tuner(None)
                times = _timer(plan, ts, stream, reps=7, graph=args.timing == "graph")
                med = statistics.median(times)
                res[name] = {"t_med_us": med * 1e6, "busbw": bus_bw(coll, size, med, n),
                             "cv": statistics.pstdev(times) / statistics.mean(times),
                             "algo": plan.info["algo_name"],
                             "proto": plan.info["proto_name"], "nchannels": plan.info["nchannels"],
                             "chunk": plan.info["chunk_elems"] * 4, "nwaves": plan.info["nwaves"]}
                plan.destroy()
            rec = {"coll": coll, "dtype": dtype, "timing": args.timing, "size": size, **{f"{k}_{kk}": vv for k, v in res.items() for kk, vv in v.items()},
                   "ratio": res["tuned"]["busbw"] / res["default"]["busbw"],
                   "ratio_ring": res["tuned_ring"]["busbw"] / res["default"]["busbw"],
                   "bad_channels_loss": 1 - res["bad_channels"]["busbw"] / res["default"]["busbw"]}
            fo.write(json.dumps(rec) + "\n")
            print(json.dumps(rec), flush=True)
            del ts


def stability(args):
    """Independent repeats of one size: fresh inputs and a fresh plan per run,
    mean / standard deviation / coefficient of variation of bus bandwidth
    (the paper's 20-run stability study, section 5.3)."""
    import torch

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    n, size, coll = args.nranks, args.size, args.coll
    # size = bytes of each rank's full buffer; AllGather / ReduceScatter
    # plans count one block of it.
    count = size // 4 if coll == "allreduce" else size // 4 // n
    out = {}
    for name, tuner, algo in (("tuned", None, "auto"), ("tuned_ring", None, "ring"),
                              ("default", "fixed_default", "auto")):
        bws = []
        for run in range(args.runs):
            g = torch.Generator(device="cuda:0").manual_seed(11438 + 200 + run)
            ts = [torch.rand(size // 4, device="cuda:0", generator=g) * 2 - 1 for _ in range(n)]
            ar.ar_set_tuner(tuner)
            plan = ar.Plan(n, count, "f32", proto="auto", algo=algo, coll=coll)
            ar.ar_set_tuner(None)
            times = _timer(plan, ts, stream, reps=1)
            # bus bandwidth: AllReduce S/t 2(N-1)/N; AllGather / ReduceScatter S/t (N-1)/N
            factor = 2.0 if coll == "allreduce" else 1.0
            bws.append(size / times[0] * factor * (n - 1) / n / 1e9)
            plan.destroy()
            del ts
        mean = statistics.mean(bws)
        sd = statistics.stdev(bws) if len(bws) > 1 else 0.0
        out[name] = {"mean_busbw": mean, "sd": sd, "cv": sd / mean, "min": min(bws), "max": max(bws),
                     "runs": len(bws)}
        print(json.dumps({"coll": coll, "size": size, "policy": name, **out[name]}), flush=True)
    with open(args.out, "a") as fo:
        fo.write(json.dumps({"coll": coll, "size": size, **out}) + "\n")


def _pct(v, q):
    v = sorted(v)
    return v[min(len(v) - 1, max(0, int(round(q * (len(v) - 1)))))]


def _stats(times_s):
    us = [t * 1e6 for t in times_s]
    mean = statistics.mean(us)
    return {"p10_us": _pct(us, 0.1), "p50_us": statistics.median(us), "p90_us": _pct(us, 0.9),
            "cv": statistics.pstdev(us) / mean if mean else 0.0}


def latency(args):
    """Small-message time per call, launched back to back from the host and
    replayed from a HIP graph that holds `--graph-runs` calls (out of place,
    so every call does the same work).  Host launches are timed through a
    bound call (`Plan.bind`: one C call per run) and, as `eager_checked`,
    through `Plan.run_oop`, which checks and marshals the buffers on every
    call."""
    import torch

    torch.cuda.set_device(0)
    n = args.nranks
    sizes = [int(s) for s in args.sizes.split(",")] if args.sizes else [1 << k for k in range(12, 23)]
    k = args.graph_runs
    with open(args.out, "a") as fo:
        for size in sizes:
            count = size // 4
            g0 = torch.Generator(device="cuda:0").manual_seed(11438 + 200)
            send = [torch.rand(count, device="cuda:0", generator=g0) * 2 - 1 for _ in range(n)]
            recv = [torch.empty(count, device="cuda:0") for _ in range(n)]
            for name, kw in (("tuned", dict(proto="auto", algo="auto")), ("ring", dict(proto="auto", algo="ring")),
                             ("direct", dict(algo="direct"))):
                plan = ar.Plan(n, count, "f32", **kw)
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                fn = plan.bind(send, recv, side)
                with torch.cuda.stream(side):
                    for _ in range(5):
                        fn()
                    side.synchronize()
                    eager, checked = [], []
                    for out, call in ((eager, fn), (checked, lambda: plan.run_oop(send, recv, side))):
                        for _ in range(7):
                            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                            e0.record(side)
                            for _ in range(k):
                                call()
                            e1.record(side)
                            e1.synchronize()
                            out.append(e0.elapsed_time(e1) / k / 1e3)
                torch.cuda.synchronize()
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph, stream=side):
                    for _ in range(k):
                        fn()
                torch.cuda.synchronize()
                graph.replay()
                torch.cuda.synchronize()
                replay = []
                for _ in range(7):
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    graph.replay()
                    e1.record()
                    e1.synchronize()
                    replay.append(e0.elapsed_time(e1) / k / 1e3)
                if plan.status() != ar.AR_OK:
                    raise RuntimeError(f"{name} {size}: plan status {plan.status()}")
                info = plan.info
                rec = {"size": size, "policy": name, "algo": info["algo_name"], "proto": info["proto_name"],
                       "nchannels": info["nchannels"], "nwaves": info["nwaves"], "runs_per_graph": k,
                       "eager": _stats(eager), "eager_checked": _stats(checked), "graph": _stats(replay)}
                fo.write(json.dumps(rec) + "\n")
                print(json.dumps(rec), flush=True)
                del graph
                plan.destroy()


def _median(v):
    return float(statistics.median(v)) if len(v) else float("nan")


def trace(args):
    """Where a ring hop's time goes, from AR_DEBUG_TRACE records (channel 0 /
    wave 0 of every rank; 100 MHz real-time stamps).  For every message a
    rank r publishes at its step j, paired with rank r+1's step j+1 that
    takes it:

        recv->issued   rank r took its input message and issued its stores
                       (LL128 / Simple: includes reading the data)
        issued->drained  those stores completed (Simple, LL128)
        drained->posted  the flag or counter store issued
        posted->taken  until rank r+1 accepted the message (visibility
                       latency plus polling)
        hop            rank r's acceptance to rank r+1's acceptance

    Medians over all pairs and runs.  The traced kernels are the builds with
    the debug hooks, which are somewhat slower than the production ones;
    `prod_us_per_hop` and `dbg_us_per_hop` give the whole-run time per hop of
    both for the same plan (graph replay, out of place)."""
    import numpy as np
    import torch

    torch.cuda.set_device(0)
    n = args.nranks
    sizes = [int(s) for s in args.sizes.split(",")]
    with open(args.out, "a") as fo:
        for proto in args.protos.split(","):
            for size in sizes:
                count = size // 4
                g0 = torch.Generator(device="cuda:0").manual_seed(11438 + 300)
                send = [torch.rand(count, device="cuda:0", generator=g0) * 2 - 1 for _ in range(n)]
                recv = [torch.empty(count, device="cuda:0") for _ in range(n)]
                flags = ar.AR_PLAN_FIFO_ONLY if args.fifo_only else 0
                kw = dict(proto=proto, nchannels=args.channels, nwaves=args.waves, flags=flags)
                if args.chunk:
                    kw["chunk_bytes"] = args.chunk
                per_hop = {}
                for label, dbg in (("prod", 0), ("dbg", ar.AR_DEBUG_TRACE)):
                    plan = ar.Plan(n, count, "f32", debug_flags=dbg, **kw)
                    buf = None
                    if dbg:
                        buf = torch.zeros(n * args.records * 8, dtype=torch.int64, device="cuda:0")
                        plan.set_trace(buf)
                    side = torch.cuda.Stream()
                    side.wait_stream(torch.cuda.current_stream())
                    t = _timer(plan, send, side, graph=True)
                    info = plan.info
                    hops = info["msgs_per_run"]  # messages of one link per run
                    per_hop[label] = statistics.median(t) / hops * 1e6
                    if not dbg:
                        plan.destroy()
                        continue
                    samples = {k: [] for k in ("recv_issued", "issued_drained", "drained_posted", "posted_taken",
                                               "hop")}
                    stale = []
                    fn = plan.bind(send, recv, side)
                    for _ in range(args.runs):
                        buf.zero_()
                        with torch.cuda.stream(side):
                            fn()
                        torch.cuda.synchronize()
                        rec = buf.cpu().numpy().view(np.uint64).reshape(n, args.records, 8).astype(np.int64)
                        nrec = int(np.count_nonzero(rec[0, :, 0]))
                        for r in range(n):
                            q = (r + 1) % n
                            for j in range(nrec - 1):
                                t_begin, t_recv, polls, t_iss, t_dr, t_post, msg, kind = rec[r, j]
                                if kind == 4 or t_post == 0:
                                    continue  # sends nothing
                                taken = rec[q, j + 1, 1]
                                if taken == 0:
                                    continue
                                samples["posted_taken"].append(taken - t_post)
                                if t_dr:
                                    samples["issued_drained"].append(t_dr - t_iss)
                                    samples["drained_posted"].append(t_post - t_dr)
                                if t_recv:
                                    samples["recv_issued"].append(t_iss - t_recv)
                                    samples["hop"].append(taken - t_recv)
                                    stale.append(1.0 if polls else 0.0)
                    if plan.status() != ar.AR_OK:
                        raise RuntimeError(f"trace {proto} {size}: plan status {plan.status()}")
                    plan.destroy()
                    row = {"proto": proto, "size": size, "nranks": n, "nchannels": info["nchannels"],
                           "nwaves": info["nwaves"], "chunk_bytes": info["chunk_elems"] * 4,
                           "nchunks": info["nchunks"], "peer_direct": info["peer_direct"],
                           "pairs": len(samples["hop"])}
                    for k, v in samples.items():
                        row[k + "_us"] = round(_median(v) / 100.0, 3)
                    row["first_look_stale"] = round(_median(stale) if not stale else sum(stale) / len(stale), 3)
                    row["prod_us_per_hop"] = round(per_hop["prod"], 3)
                    row["dbg_us_per_hop"] = round(per_hop["dbg"], 3)
                    fo.write(json.dumps(row) + "\n")
                    print(json.dumps(row), flush=True)


def _to_device(x, dtype):
    """(N, count) numpy array (float32, or uint16 bf16 bits) -> one device tensor per rank."""
    import numpy as np
    import torch

    if dtype == "f32":
        return [torch.from_numpy(np.ascontiguousarray(x[r])).to("cuda:0") for r in range(x.shape[0])]
    return [torch.from_numpy(np.ascontiguousarray(x[r]).view(np.int16)).view(torch.bfloat16).to("cuda:0")
            for r in range(x.shape[0])]


def _config_points(name):
    """Plan settings of each measured point of the named workload."""
    import workloads

    wl = workloads.WORKLOADS[name]
    if name == "D1":
        return wl, [dict(proto="simple", nchannels=1, chunk_bytes=1024)]
    if name == "D2":
        return wl, [dict(proto=p, nchannels=c) for p in wl.protos for c in wl.channels]
    if name == "D3":
        return wl, [dict(proto="simple", nchannels=c, chunk_bytes=k) for k in wl.chunks for c in wl.channels]
    if name == "D5":
        return wl, ([dict(proto=p, nchannels=c) for p in wl.protos for c in wl.channels] +
                    [dict(proto="simple", nchannels=c, flags=ar.AR_PLAN_FIFO_ONLY) for c in wl.channels])
    raise ValueError(name)


def configs(args):
    """The named workloads at their stated settings: time per call (median,
    p10, p90, CV over 7 repeats), algBW / busBW, the fraction of 8 TB/s on
    the ring-byte and compulsory-byte bases, and ring bytes per element."""
    import torch

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    peak = 8000.0  # GB/s
    with open(args.out, "a") as fo:
        for name in args.names.split(","):
            wl, points = _config_points(name)
            n, count, dtype = wl.nranks, wl.count, wl.dtype
            size = wl.bytes_per_rank
            ts = _to_device(wl.draw(), dtype)
            for cfg in points:
                plan = ar.Plan(n, count, dtype, **cfg)
                times = _timer(plan, ts, stream, reps=7, warm=5)
                info = plan.info
                st = _stats(times)
                t = st["p50_us"] * 1e-6
                rb = ar.ring_bytes(size, n, dtype, info["proto_name"], peer_direct=bool(info["peer_direct"]))
                cb = ar.compulsory_bytes(size, n)
                rec = {"workload": name, "size": size, "dtype": dtype, **cfg, "proto": info["proto_name"],
                       "peer_direct": info["peer_direct"],
                       "nchannels_eff": info["nchannels"], "chunk_eff": info["chunk_elems"] * (4 if dtype == "f32" else 2),
                       "nwaves": info["nwaves"], "nchunks": info["nchunks"], **st,
                       "algbw": ar.alg_bandwidth(size, t), "busbw": ar.bus_bandwidth(size, t, n),
                       "hbm_frac_ring": rb / t / 1e9 / peak, "hbm_frac_comp": cb / t / 1e9 / peak,
                       "ring_bytes_per_elem": rb / count}
                if name == "D1":
                    graph = torch.cuda.CUDAGraph()
                    side = torch.cuda.Stream()
                    side.wait_stream(torch.cuda.current_stream())
                    run = _runner(plan, ts)
                    with torch.cuda.stream(side):
                        run(side)
                    torch.cuda.synchronize()
                    with torch.cuda.graph(graph, stream=side):
                        for _ in range(100):
                            run(side)
                    graph.replay()
                    torch.cuda.synchronize()
                    rep = []
                    for _ in range(7):
                        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                        e0.record()
                        graph.replay()
                        e1.record()
                        e1.synchronize()
                        rep.append(e0.elapsed_time(e1) / 100 / 1e3)
                    rec["graph"] = _stats(rep)
                    del graph
                if plan.status() != ar.AR_OK:
                    raise RuntimeError(f"{name} {cfg}: plan status {plan.status()}")
                plan.destroy()
                fo.write(json.dumps(rec) + "\n")
                fo.flush()
                print(json.dumps(rec), flush=True)
            del ts
            torch.cuda.empty_cache()


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    m = sub.add_parser("measure")
    m.add_argument("--out", required=True)
    m.add_argument("--sizes", default="")
    m.add_argument("--nranks", type=int, default=8)
    m.add_argument("--algo", default="", help="measure only this algorithm (ring or direct)")
    m.add_argument("--coll", default="allreduce", choices=("allreduce", "allgather", "reducescatter"))
    m.add_argument("--dtype", default="f32", choices=("f32", "bf16"))
    m.add_argument("--timing", default="graph", choices=("graph", "eager"))
    t = sub.add_parser("table")
    t.add_argument("jsonl", nargs="+")
    t.add_argument("--emit", default="")
    t.add_argument("--validated", nargs="*", default=[],
                   help="`validate` outputs: ring rows within 2 %% of the default there defer to it")
    v = sub.add_parser("validate")
    v.add_argument("--out", required=True)
    v.add_argument("--nranks", type=int, default=8)
    v.add_argument("--sizes", default="")
    v.add_argument("--coll", default="allreduce", choices=("allreduce", "allgather", "reducescatter"))
    v.add_argument("--dtype", default="f32", choices=("f32", "bf16"))
    v.add_argument("--timing", default="eager", choices=("graph", "eager"))
    st = sub.add_parser("stability")
    st.add_argument("--out", required=True)
    st.add_argument("--size", type=int, default=128 << 20)
    st.add_argument("--runs", type=int, default=20)
    st.add_argument("--nranks", type=int, default=8)
    st.add_argument("--coll", default="allreduce", choices=("allreduce", "allgather", "reducescatter"))
    co = sub.add_parser("configs")
    co.add_argument("--out", required=True)
    co.add_argument("--names", default="D1,D2,D3,D5")
    la = sub.add_parser("latency")
    la.add_argument("--out", required=True)
    la.add_argument("--sizes", default="")
    la.add_argument("--nranks", type=int, default=8)
    la.add_argument("--graph-runs", type=int, default=100)
    tr = sub.add_parser("trace")
    tr.add_argument("--out", required=True)
    tr.add_argument("--protos", default="simple,ll,ll128")
    tr.add_argument("--sizes", default="4096,65536,1048576")
    tr.add_argument("--nranks", type=int, default=8)
    tr.add_argument("--channels", type=int, default=1)
    tr.add_argument("--waves", type=int, default=1)
    tr.add_argument("--chunk", type=int, default=0)
    tr.add_argument("--records", type=int, default=4096, help="trace records kept per rank")
    tr.add_argument("--runs", type=int, default=20)
    tr.add_argument("--fifo-only", action="store_true")
    args = ap.parse_args(argv)
    {"measure": measure, "table": table_cmd, "validate": validate, "stability": stability,
     "latency": latency, "configs": configs, "trace": trace}[args.cmd](args)


if __name__ == "__main__":
    sys.exit(main())
