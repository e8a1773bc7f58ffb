"""Selection of the built-in tuner tables from sweep rows (host logic, no
GPU): the highest median bus bandwidth wins; rows within 2 % of it are ties,
broken by fewer channels, fewer wire bytes (Simple < LL128 < LL), smaller
chunk, then the higher bandwidth; channels and chunk count as the plan
resolved them; a size defers to the fixed default when the default is
within 2 %; the direct algorithm is taken when it is within 2 % of the best
ring choice or faster; AllReduce rows of each data type make their own
table."""
from __future__ import annotations

import paper_2603_11438_amd as ar
from paper_2603_11438_amd import sweep

SIZE = 1 << 24


def ring(proto, c, chunk, w, bw, size=SIZE, chunk_eff=None, parts_eff=None, dtype="f32"):
    return {"coll": "allreduce", "dtype": dtype, "size": size, "algo": "ring", "proto": proto, "nchannels": c,
            "chunk_bytes": chunk, "nwaves": w, "busbw": bw, "chunk_eff": chunk if chunk_eff is None else chunk_eff,
            "parts_eff": c if parts_eff is None else parts_eff}


def direct(parts, w, bw, parts_eff=None, size=SIZE, dtype="f32"):
    return {"coll": "allreduce", "dtype": dtype, "size": size, "algo": "direct", "proto": "simple", "nchannels": parts,
            "nwaves": w, "direct_unroll": 1, "busbw": bw, "parts_eff": parts if parts_eff is None else parts_eff,
            "chunk_bytes": 0, "chunk_eff": 0}


def pick(rows):
    return sweep.select_ring(rows)[SIZE]


def test_clear_winner():
    assert pick([ring("simple", 32, 65536, 4, 300.0), ring("ll", 8, 4096, 2, 250.0)])["busbw"] == 300.0


def test_ties_prefer_fewer_channels_then_wire_bytes_then_chunk_then_bandwidth():
    rows = [ring("simple", 32, 65536, 4, 300.0), ring("simple", 16, 65536, 4, 295.0)]
    assert pick(rows)["nchannels"] == 16                       # 295 is within 2 % of 300
    rows = [ring("ll", 16, 4096, 4, 300.0), ring("simple", 16, 65536, 4, 296.0)]
    assert pick(rows)["proto"] == "simple"                      # fewer wire bytes
    rows = [ring("ll128", 16, 61440, 4, 300.0), ring("ll", 16, 4096, 4, 299.0)]
    assert pick(rows)["proto"] == "ll128"
    rows = [ring("simple", 16, 262144, 4, 300.0), ring("simple", 16, 65536, 8, 297.0)]
    assert pick(rows)["chunk_bytes"] == 65536                   # smaller chunk
    rows = [ring("simple", 16, 65536, 4, 297.0), ring("simple", 16, 65536, 8, 300.0)]
    assert pick(rows)["nwaves"] == 8                            # then the higher bandwidth
    rows = [ring("simple", 32, 65536, 4, 300.0), ring("simple", 16, 65536, 4, 290.0)]
    assert pick(rows)["nchannels"] == 32                        # 290 is outside the band


def test_ties_compare_the_resolved_geometry():
    # a chunk past a channel's share resolves to the share: equal geometry,
    # so the bandwidth decides, not the nominal chunk
    rows = [ring("simple", 16, 1 << 20, 4, 300.0, chunk_eff=131072), ring("simple", 16, 131072, 4, 297.0)]
    assert pick(rows)["busbw"] == 300.0


def test_direct_ties_compare_resolved_parts():
    rows = [ring("simple", 64, 65536, 4, 300.0), direct(0, 1, 600.0, parts_eff=256), direct(128, 1, 595.0)]
    row = sweep.select(rows)[SIZE]
    assert row["algo"] == "direct"
    assert row["direct"]["parts_eff"] == 128                    # not the size rule's "0" (= 256)


def test_algorithm_column():
    rows = [ring("simple", 64, 65536, 4, 300.0), direct(64, 1, 295.0)]
    assert sweep.select(rows)[SIZE]["algo"] == "direct"         # within 2 %: fewer bytes
    rows = [ring("simple", 64, 65536, 4, 300.0), direct(64, 1, 280.0)]
    assert sweep.select(rows)[SIZE]["algo"] == "ring"


def test_defers_to_the_fixed_default_within_the_band():
    count = SIZE // 4
    g = ar.ar_plan_geometry(ar.make_desc(8, count, "f32", "simple", 16, sweep.DEFAULT_CHUNK,
                                         nwaves=sweep.DEFAULT_WAVES))
    dflt = ring("simple", 16, sweep.DEFAULT_CHUNK, sweep.DEFAULT_WAVES, 296.0, chunk_eff=g["chunk_elems"] * 4)
    assert pick([ring("simple", 32, 65536, 4, 300.0), dflt])["proto"] == "default"
    dflt = dict(dflt, busbw=280.0)
    assert pick([ring("simple", 32, 65536, 4, 300.0), dflt])["nchannels"] == 32


def test_each_dtype_makes_its_own_allreduce_table(tmp_path):
    rows = [ring("simple", 32, 65536, 4, 300.0), direct(128, 1, 600.0),
            ring("simple", 64, 65536, 8, 260.0, dtype="bf16"), direct(96, 2, 500.0, dtype="bf16")]
    import json
    src = tmp_path / "rows.jsonl"
    src.write_text("\n".join(json.dumps(r) for r in rows) + "\n")
    out = tmp_path / "table.inc"
    sweep.table_cmd(type("A", (), {"jsonl": [str(src)], "emit": str(out)})())
    text = out.read_text()
    f32 = text.split("kTableAllReduce[]")[1].split("};")[0]
    bf16 = text.split("kTableAllReduceBf16[]")[1].split("};")[0]
    assert "AR_PROTO_SIMPLE, 32, 65536, 4, AR_ALGO_DIRECT, 128, 1, 1" in f32
    assert "AR_PROTO_SIMPLE, 64, 65536, 8, AR_ALGO_DIRECT, 96, 2, 1" in bf16
    # collectives without rows keep a row that defers to the default
    assert "not measured" in text.split("kTableReduceScatter[]")[1].split("};")[0]


def test_bf16_table_falls_back_to_the_fp32_rows(tmp_path):
    import json
    src = tmp_path / "rows.jsonl"
    src.write_text(json.dumps(ring("simple", 32, 65536, 4, 300.0)) + "\n")
    out = tmp_path / "table.inc"
    sweep.table_cmd(type("A", (), {"jsonl": [str(src)], "emit": str(out)})())
    text = out.read_text()
    f32 = text.split("kTableAllReduce[]")[1].split("};")[0]
    bf16 = text.split("kTableAllReduceBf16[]")[1].split("};")[0]
    assert f32.strip() and f32 == bf16


def test_validated_ratio_within_tie_defers_to_default():
    """A ring choice made on the sweep's repeats that validates within 2 % of
    the fixed default on fresh repeats defers to the default; one that
    validates clearly faster keeps its row."""
    rows = [ring("ll", 16, 4096, 4, 300.0), ring("simple", 32, 65536, 4, 250.0)]
    keep = sweep.select(rows, validated={SIZE: 1.25})[SIZE]["ring"]
    assert keep["proto"] == "ll"
    dropped = sweep.select(rows, validated={SIZE: 0.99})[SIZE]["ring"]
    assert dropped["proto"] == "default" and dropped["validated_ratio"] == 0.99
    edge = sweep.select(rows, validated={SIZE: 1.019})[SIZE]["ring"]
    assert edge["proto"] == "default"
    # sizes without a validation keep the sweep's choice
    assert sweep.select(rows, validated={SIZE * 2: 0.5})[SIZE]["ring"]["proto"] == "ll"
    # the emitted row leaves the ring columns to the default
    text = sweep.emit_one({SIZE: sweep.select(rows, validated={SIZE: 0.99})[SIZE]}, ("allreduce", "f32"))
    assert "{24, AR_PROTO_AUTO, 0, 0, 0," in text
