// Tuner, plan geometry and error strings of libar: host-only C++ with no
// HIP dependency, so it also builds (and is sanitizer-tested) with g++.
//
// Tuner semantics follow the paper's policy model (section 3.3: a policy
// reads collective type, message size and rank count and writes algorithm,
// protocol and channel count; section 4: outputs that cannot be honoured
// fall back to the library's own choice, and the requested channel count is
// clamped to the maximum the library passes in; section 5.3: the
// size-aware policy picks one ring protocol for mid sizes and another for
// large sizes).
#include <atomic>
#include <chrono>
#include <new>
#include <thread>
#include <stddef.h>
#include <stdint.h>

#include "ar.h"
#include "ar_internal.h"

namespace ar {

namespace {

thread_local int g_last_error = AR_OK;

struct TableRow {
    int log2_bytes;
    int proto;         // ring choice for this size ...
    int nchannels;
    size_t chunk_bytes;
    int nwaves;
    int algo;          // ... and the algorithm to run (AUTO = the ring)
    int direct_parts;  // direct algorithm's workgroups per segment (0 = auto)
    int direct_nwaves; // direct algorithm's waves per workgroup (0 = default)
    int direct_unroll; // direct algorithm's units per thread and iteration (0 = by size)
};

#include "tuner_table.inc"

template <size_t K>
constexpr int rows_of(const TableRow (&)[K]) { return (int)K; }

constexpr int kDefaultProto = AR_PROTO_SIMPLE;
constexpr int kDefaultChannels = 16;
constexpr size_t kMaxChunkBytes = 64u << 20;
constexpr size_t kMinChunkBytes = 16;

bool valid_proto(int p) { return p == AR_PROTO_LL || p == AR_PROTO_LL128 || p == AR_PROTO_SIMPLE; }
bool valid_algo(int a) { return a == AR_ALGO_AUTO || a == AR_ALGO_RING || a == AR_ALGO_DIRECT; }

// The active tuner is one atomic pointer to an immutable slot (paper section
// 4, hot reload: an atomic function-pointer swap; a call already in progress
// finishes with the old policy, the next call uses the new one).  Each slot
// counts the decisions running through it, so a reload can wait until the
// replaced slot has drained; slots are never freed (a late reader may still
// touch the counter of a replaced slot), which costs one small allocation
// per reload.
struct TunerSlot {
    ar_tuner_fn fn;
    void *user;
    std::atomic<int64_t> inflight{0};
};

TunerSlot g_builtin_slot{ar_tuner_table, nullptr};
std::atomic<TunerSlot *> g_active{&g_builtin_slot};

uint64_t now_ns()
{
    return (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
               std::chrono::steady_clock::now().time_since_epoch())
        .count();
}

// Pin the active slot for one decision.  The increment and the re-check are
// sequentially consistent, pairing with the exchange and the drain load in
// install(): either the reload sees this reader in `inflight`, or this reader
// sees the new slot and backs off.
TunerSlot *pin_active()
{
    for (;;) {
        TunerSlot *s = g_active.load(std::memory_order_seq_cst);
        s->inflight.fetch_add(1, std::memory_order_seq_cst);
        if (g_active.load(std::memory_order_seq_cst) == s) return s;
        s->inflight.fetch_sub(1, std::memory_order_seq_cst);
    }
}

void unpin(TunerSlot *s) { s->inflight.fetch_sub(1, std::memory_order_seq_cst); }

bool out_valid(int rc, const ar_tune_out &o)
{
    if (rc != 0) return false;
    if (!valid_algo(o.algo)) return false;
    if (o.proto != AR_PROTO_AUTO && !valid_proto(o.proto)) return false;
    if (o.nchannels < 0 || o.nwaves < 0 || o.nwaves > AR_MAX_WAVES) return false;
    if (o.direct_parts < 0 || o.direct_nwaves < 0 || o.direct_nwaves > AR_MAX_WAVES) return false;
    if (o.direct_unroll < 0 || o.direct_unroll > 2) return false;
    return o.chunk_bytes <= kMaxChunkBytes;
}

// Load-time check of a candidate tuner: call it on a grid of contexts and
// reject it if any answer is malformed (paper section 3.1, T1: verify once
// at load time; a policy that is well-formed but makes poor choices still
// passes, as in section 5.3).
int probe_tuner(ar_tuner_fn fn, void *user, uint64_t *probes)
{
    static const size_t sizes[] = {0, 1, 4096, 65536, 1u << 20, 4u << 20, 32u << 20, 128u << 20, 1u << 30};
    static const int ranks[] = {1, 2, 8, 16};
    static const int maxch[] = {1, 64, AR_MAX_CHANNELS};
    uint64_t n = 0;
    for (size_t sz : sizes)
        for (int nr : ranks)
            for (int dt = 0; dt < 2; ++dt)
                for (int mc : maxch) {
                    ar_tune_ctx c = {AR_COLL_ALLREDUCE, sz, nr, dt, mc, 0};
                    ar_tune_out o = {AR_PROTO_AUTO, 0, 0, 0, AR_ALGO_AUTO, 0, 0};
                    int rc = fn(&c, &o, user);
                    ++n;
                    if (!out_valid(rc, o)) {
                        if (probes) *probes = n;
                        return AR_ERR_ARG;
                    }
                }
    if (probes) *probes = n;
    return AR_OK;
}

int install(ar_tuner_fn fn, void *user, bool validate, ar_reload_stats *st)
{
    ar_reload_stats z = {0, 0, 0, 0};
    uint64_t t0 = now_ns();
    TunerSlot *ns = &g_builtin_slot;
    if (fn) {
        if (validate) {
            int rc = probe_tuner(fn, user, &z.probes);
            if (rc != AR_OK) {
                z.validate_ns = now_ns() - t0;
                if (st) *st = z;
                return rc;
            }
        }
        ns = new (std::nothrow) TunerSlot{fn, user};
        if (!ns) return AR_ERR_NOMEM;
    }
    uint64_t t1 = now_ns();
    TunerSlot *old = g_active.exchange(ns, std::memory_order_seq_cst);
    uint64_t t2 = now_ns();
    // Drain: decisions that pinned the old slot finish before we return, so
    // the caller may release the old tuner's code and data afterwards.
    while (old != ns && old->inflight.load(std::memory_order_seq_cst) != 0) std::this_thread::yield();
    uint64_t t3 = now_ns();
    z.validate_ns = t1 - t0;
    z.swap_ns = t2 - t1;
    z.drain_ns = t3 - t2;
    if (st) *st = z;
    return AR_OK;
}

inline uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }
inline uint64_t round_up(uint64_t a, uint64_t b) { return ceil_div(a, b) * b; }

int clamp_int(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

size_t clamp_chunk(size_t c)
{
    if (c < kMinChunkBytes) c = kMinChunkBytes;
    if (c > kMaxChunkBytes) c = kMaxChunkBytes;
    return c / 16 * 16;
}

}  // namespace

void set_last_error(int code) { g_last_error = code; }

int default_nwaves(int proto)
{
    (void)proto;
    return 4;
}

int default_depth(int proto) { return proto == AR_PROTO_SIMPLE ? 2 : 4; }
constexpr int kMaxDepth = 16;
constexpr uint64_t kSmallFifoBytes = 4ull << 20;

// Direct algorithm: units (16 bytes of data) per thread per iteration, and
// the largest grid it is sized to (8 workgroups per CU on 256 CUs).
// Direct algorithm: two units per thread and iteration up to this many bytes
// per rank, one above (measured on MI355X: two keep more loads in flight
// while the data is cache-resident, one streams faster from HBM).
constexpr uint64_t kDirectUnrollBytes = 8ull << 20;
constexpr uint64_t kDirectMaxGrid = 2048;

size_t default_chunk_bytes(int proto)
{
    switch (proto) {
    case AR_PROTO_LL: return 16u << 10;
    case AR_PROTO_LL128: return 60u << 10;
    default: return 256u << 10;
    }
}

// Geometry of the direct algorithm: a group of `parts` workgroups per
// segment, each striding over the segment's 16-byte units.
int resolve_direct(const ar_plan_desc *d, const ar_tune_out *t, ar_plan_info *out)
{
    const uint64_t e = d->dtype == AR_FLOAT32 ? 4 : 2;
    const uint64_t A = 16 / e;
    const uint64_t N = (uint64_t)d->nranks;
    int nw = d->nwaves ? d->nwaves : (t && t->direct_nwaves ? t->direct_nwaves : 4);
    const uint64_t full_bytes = d->count * e * (d->coll == AR_COLL_ALLREDUCE ? 1 : N);
    int unroll = d->direct_unroll ? d->direct_unroll : (t && t->direct_unroll ? t->direct_unroll : 0);
    if (unroll == 0) unroll = full_bytes <= kDirectUnrollBytes ? 2 : 1;
    if (d->nranks > 8) unroll = 1;  // the 9..16-rank kernel keeps one unit per thread
    ar_plan_info g = {};
    g.algo = AR_ALGO_DIRECT;
    g.direct_unroll = unroll;
    g.coll = d->coll;
    g.proto = AR_PROTO_AUTO;
    g.nranks = d->nranks;
    g.dtype = d->dtype;
    g.nwaves = nw;
    g.placement = d->placement;
    g.count = d->count;
    g.block = 64 * nw;
    g.seg_elems = d->coll == AR_COLL_ALLREDUCE ? round_up(ceil_div(d->count, N), A) : d->count;
    if (N == 1 || d->count == 0) {
        g.grid = 0;
        *out = g;
        return AR_OK;
    }
    const uint64_t seg_units = ceil_div(g.seg_elems, A);
    uint64_t parts = (uint64_t)(d->nchannels ? d->nchannels : (t ? t->direct_parts : 0));
    if (parts == 0) {
        parts = ceil_div(seg_units, 64 * (uint64_t)nw * (uint64_t)unroll);
        uint64_t cap = kDirectMaxGrid / N;
        if (cap < 1) cap = 1;
        if (parts > cap) parts = cap;
        if (parts < 1) parts = 1;
    }
    g.nchannels = (int)parts;
    g.grid = (int)(parts * N);
    g.chan_elems = round_up(ceil_div(g.seg_elems, parts), A);
    *out = g;
    return AR_OK;
}

int resolve_geometry(const ar_plan_desc *d, int max_channels, ar_plan_info *out)
{
    if (!d || !out) return AR_ERR_ARG;
    if (d->nranks < 1 || d->nranks > AR_MAX_RANKS) return AR_ERR_ARG;
    if (d->dtype != AR_FLOAT32 && d->dtype != AR_BFLOAT16) return AR_ERR_ARG;
    if (d->proto != AR_PROTO_AUTO && !valid_proto(d->proto)) return AR_ERR_ARG;
    if (d->nchannels < 0 || d->nchannels > AR_MAX_CHANNELS) return AR_ERR_ARG;
    if (d->fifo_depth != 0 && (d->fifo_depth < 2 || d->fifo_depth > kMaxDepth)) return AR_ERR_ARG;
    if (d->nwaves < 0 || d->nwaves > AR_MAX_WAVES) return AR_ERR_ARG;
    if (d->direct_unroll < 0 || d->direct_unroll > 2) return AR_ERR_ARG;
    if (d->placement != AR_PLACE_RANK_SPREAD && d->placement != AR_PLACE_CHANNEL_LOCAL) return AR_ERR_ARG;
    if (d->chunk_bytes > kMaxChunkBytes) return AR_ERR_ARG;
    if (d->flags & ~(uint32_t)(AR_PLAN_PROFILE | AR_PLAN_FIFO_ONLY | AR_PLAN_LL128_ORDERED)) return AR_ERR_ARG;
    if (!valid_algo(d->algo)) return AR_ERR_ARG;
    if (d->coll != AR_COLL_ALLREDUCE && d->coll != AR_COLL_REDUCESCATTER && d->coll != AR_COLL_ALLGATHER)
        return AR_ERR_ARG;
    if (max_channels < 1) max_channels = 1;
    if (max_channels > AR_MAX_CHANNELS) max_channels = AR_MAX_CHANNELS;

    const uint64_t e = d->dtype == AR_FLOAT32 ? 4 : 2;
    const uint64_t A = 16 / e;
    // Per-rank byte counts stay below 2^46 so every byte offset fits easily.
    if (d->count > (1ull << 44) / (uint64_t)d->nranks) return AR_ERR_ARG;
    if (d->coll != AR_COLL_ALLREDUCE && d->count % A != 0) return AR_ERR_UNSUPPORTED;
    // Bytes of the full per-rank buffer (what the tuner sizes its decision by).
    const uint64_t full_bytes = d->count * e * (d->coll == AR_COLL_ALLREDUCE ? 1 : (uint64_t)d->nranks);

    // A requested protocol implies the ring.
    int algo = d->algo;
    if (algo == AR_ALGO_AUTO && d->proto != AR_PROTO_AUTO) algo = AR_ALGO_RING;
    if (algo == AR_ALGO_DIRECT && d->proto != AR_PROTO_AUTO) return AR_ERR_ARG;
    int proto = d->proto, nch = d->nchannels, nw = d->nwaves;
    size_t chunk = d->chunk_bytes;
    // One decision per plan: the tuner is asked at most once.
    const bool ring_needs_tuner = proto == AR_PROTO_AUTO || nch == 0 || chunk == 0 || nw == 0;
    const bool direct_needs_tuner = nch == 0 || nw == 0;
    ar_tune_out t;
    bool have_t = false;
    if (algo == AR_ALGO_AUTO || (algo == AR_ALGO_RING && ring_needs_tuner) ||
        (algo == AR_ALGO_DIRECT && direct_needs_tuner)) {
        ar_tune_ctx ctx = {d->coll, (size_t)full_bytes, d->nranks, d->dtype, max_channels, d->comm_id};
        int rc = ar_tune(&ctx, &t);
        if (rc != AR_OK) return rc;
        have_t = true;
        if (algo == AR_ALGO_AUTO) algo = t.algo;
        if (algo == AR_ALGO_RING) {
            if (proto == AR_PROTO_AUTO) {
                proto = t.proto;
                // Channels, chunk and waves from the tuner belong to its protocol.
                if (nch == 0) nch = t.nchannels;
                if (chunk == 0) chunk = t.chunk_bytes;
                if (nw == 0) nw = t.nwaves;
            } else {
                if (nch == 0) nch = t.proto == proto ? t.nchannels : clamp_int(kDefaultChannels, 1, max_channels);
                if (chunk == 0) chunk = t.proto == proto ? t.chunk_bytes : default_chunk_bytes(proto);
                if (nw == 0) nw = t.proto == proto ? t.nwaves : default_nwaves(proto);
            }
        }
    }
    if (algo == AR_ALGO_DIRECT) return resolve_direct(d, have_t ? &t : nullptr, out);
    // Ring workgroups wait on each other, so they must all be resident.
    if (d->nchannels > max_channels) return AR_ERR_OCCUPANCY;
    chunk = clamp_chunk(chunk);

    ar_plan_info g = {};
    g.algo = AR_ALGO_RING;
    g.coll = d->coll;
    g.nranks = d->nranks;
    g.dtype = d->dtype;
    g.proto = proto;
    g.nchannels = nch;
    g.nwaves = nw;
    g.placement = d->placement;
    g.count = d->count;
    g.block = 64 * nw;
    // Peer-direct mode: reduction chains start with a peer read (and the
    // Simple all-gather writes into the next rank's output);
    // AR_PLAN_FIFO_ONLY plans keep every hop in the FIFOs.
    g.peer_direct = !(d->flags & AR_PLAN_FIFO_ONLY);

    const uint64_t N = (uint64_t)d->nranks;
    g.seg_elems = d->coll == AR_COLL_ALLREDUCE ? round_up(ceil_div(d->count, N), A) : d->count;
    if (N == 1 || d->count == 0) {
        // Nothing moves between ranks: no FIFOs, no launch of the ring kernel.
        g.grid = 0;
        *out = g;
        return AR_OK;
    }
    g.grid = nch * d->nranks;
    g.chan_elems = round_up(ceil_div(g.seg_elems, (uint64_t)nch), A);
    uint64_t ck = round_up(chunk / e, A);
    if (ck < A) ck = A;
    if (ck > g.chan_elems) ck = g.chan_elems;
    g.chunk_elems = ck;
    g.nchunks = ceil_div(g.chan_elems, ck);
    g.wave_elems = round_up(ceil_div(ck, (uint64_t)nw), A);

    // Reduce-scatter partials are fp32 on the wire for both dtypes, so a slot
    // is sized for wave_elems fp32 values in the protocol's line format.
    uint64_t slot;
    switch (proto) {
    case AR_PROTO_LL: slot = g.wave_elems * 8; break;          // 4 B data + 4 B flag
    case AR_PROTO_LL128: slot = ceil_div(g.wave_elems * 4, 120) * 128; break;
    default: slot = g.wave_elems * 4; break;
    }
    g.slot_bytes = round_up(slot, 256);
    const uint64_t conns = (uint64_t)nch * N * (uint64_t)nw;
    // Messages per connection: 2N-2 per chunk (AllReduce) or N-1; in the
    // peer-direct mode a reduction chain starts with a peer read, one
    // message fewer.
    g.msgs_per_run = g.nchunks * ((d->coll == AR_COLL_ALLREDUCE ? 2 * N - 2 : N - 1) -
                                  (g.peer_direct && d->coll != AR_COLL_ALLGATHER ? 1 : 0));
    // Default depth: the protocol's, doubled (up to kMaxDepth) while a run
    // has more messages than slots and the FIFO stays within
    // kSmallFifoBytes.  A latency-bound run then finds its slots free from
    // the head value read at kernel start instead of reading the receiver's
    // head counter again, a round trip, every few messages.
    int depth = d->fifo_depth;
    if (depth == 0) {
        depth = default_depth(proto);
        while (depth < kMaxDepth && (uint64_t)depth < g.msgs_per_run &&
               conns * (uint64_t)(2 * depth) * g.slot_bytes <= kSmallFifoBytes)
            depth *= 2;
    }
    g.fifo_depth = depth;
    g.fifo_bytes = conns * (uint64_t)depth * g.slot_bytes;
    g.flag_bytes = conns * kConnFlagU64 * 8 + kCtlU32 * 4;

    // Wire bytes actually written per run.  AllReduce: each element crosses
    // 2(N-1) links, N-1 as an fp32 partial and N-1 as a finished value;
    // ReduceScatter: each of N blocks crosses N-1 links as fp32 partials;
    // AllGather: each of N blocks crosses N-1 links as data.
    const double ag_e = (double)e;
    double rs_bytes = 0, ag_bytes = 0, peer_bytes = 0;
    // In the peer-direct mode the first link of a chain carries the chain
    // start's input in the data type (a peer read, without line flags), not
    // a partial.
    const double rs_link = g.peer_direct ? 4.0 * (double)(N - 2) : 4.0 * (double)(N - 1);
    const double rs_peer = g.peer_direct ? (double)e : 0.0;
    if (d->coll == AR_COLL_ALLREDUCE) {
        rs_bytes = (double)d->count * rs_link;
        peer_bytes = (double)d->count * rs_peer;
        ag_bytes = (double)d->count * ag_e * (double)(N - 1);
    } else if (d->coll == AR_COLL_REDUCESCATTER) {
        rs_bytes = (double)d->count * (double)N * rs_link;
        peer_bytes = (double)d->count * (double)N * rs_peer;
    } else {
        ag_bytes = (double)d->count * (double)N * ag_e * (double)(N - 1);
    }
    double w = proto == AR_PROTO_LL ? 2.0 : (proto == AR_PROTO_LL128 ? 128.0 / 120.0 : 1.0);
    g.wire_bytes_per_run = (uint64_t)((rs_bytes + ag_bytes) * w + peer_bytes);

    // Sanity limits: 32-bit byte offsets inside a slot, bounded FIFO memory.
    if (g.slot_bytes > (1ull << 31)) return AR_ERR_ARG;
    if (g.fifo_bytes > (16ull << 30)) return AR_ERR_ARG;
    // LL flags repeat every 2^32 - 2 messages; a stale line in a slot is at
    // most depth * msgs_per_run messages old, which must stay below that.
    if (proto == AR_PROTO_LL && g.msgs_per_run * (uint64_t)depth >= (1ull << 31)) return AR_ERR_UNSUPPORTED;
    *out = g;
    return AR_OK;
}

}  // namespace ar

using namespace ar;

extern "C" {

int ar_tuner_fixed_default(const ar_tune_ctx *ctx, ar_tune_out *out, void *user)
{
    (void)user;
    if (!ctx || !out) return -1;
    out->proto = kDefaultProto;
    out->nchannels = kDefaultChannels;
    out->chunk_bytes = 0;
    out->nwaves = 0;
    out->algo = AR_ALGO_RING;
    out->direct_parts = 0;
    out->direct_nwaves = 0;
    out->direct_unroll = 0;
    return 0;
}

int ar_tuner_noop(const ar_tune_ctx *ctx, ar_tune_out *out, void *user)
{
    (void)ctx;
    (void)user;
    if (!out) return -1;
    out->proto = AR_PROTO_AUTO;
    out->nchannels = 0;
    out->chunk_bytes = 0;
    out->nwaves = 0;
    out->algo = AR_ALGO_AUTO;
    out->direct_parts = 0;
    out->direct_nwaves = 0;
    out->direct_unroll = 0;
    return 0;
}

// The table rows were measured with kTableRanks ranks.  A launch has
// nchannels * N ring workgroups (direct: parts * N), so for another rank
// count N a row's channel and part counts are scaled by kTableRanks / N:
// the grid keeps the workgroup count the row was measured with.  0 (the
// library's own rule) stays 0.
constexpr int kTableRanks = 8;

static int scale_to_ranks(int v, int nranks)
{
    if (v <= 0 || nranks <= 0 || nranks == kTableRanks) return v;
    const int s = (v * kTableRanks + nranks / 2) / nranks;
    return s < 1 ? 1 : s;
}

int ar_tuner_table(const ar_tune_ctx *ctx, ar_tune_out *out, void *user)
{
    (void)user;
    if (!ctx || !out) return -1;
    const TableRow *table;
    int nrows;
    switch (ctx->coll) {
    case AR_COLL_ALLREDUCE:
        // bf16 reduce-scatter hops carry fp32 partials, so the best
        // geometry moves with the data type: every collective has a table per type
        if (ctx->dtype == AR_BFLOAT16) {
            table = kTableAllReduceBf16;
            nrows = rows_of(kTableAllReduceBf16);
        } else {
            table = kTableAllReduce;
            nrows = rows_of(kTableAllReduce);
        }
        break;
    case AR_COLL_REDUCESCATTER:
        if (ctx->dtype == AR_BFLOAT16) {
            table = kTableReduceScatterBf16;
            nrows = rows_of(kTableReduceScatterBf16);
        } else {
            table = kTableReduceScatter;
            nrows = rows_of(kTableReduceScatter);
        }
        break;
    case AR_COLL_ALLGATHER:
        if (ctx->dtype == AR_BFLOAT16) {
            table = kTableAllGatherBf16;
            nrows = rows_of(kTableAllGatherBf16);
        } else {
            table = kTableAllGather;
            nrows = rows_of(kTableAllGather);
        }
        break;
    default: return ar_tuner_noop(ctx, out, nullptr);  // not tabulated: defer to the default
    }
    int lg = 0;
    while (lg < 63 && (1ull << lg) < (unsigned long long)ctx->msg_bytes) ++lg;
    const TableRow *row = &table[0];
    for (int i = 0; i < nrows; ++i) {
        row = &table[i];
        if (table[i].log2_bytes >= lg) break;
    }
    out->proto = row->proto;
    out->nchannels = scale_to_ranks(row->nchannels, ctx->nranks);
    out->chunk_bytes = row->chunk_bytes;
    out->nwaves = row->nwaves;
    out->algo = row->algo;
    out->direct_parts = scale_to_ranks(row->direct_parts, ctx->nranks);
    out->direct_nwaves = row->direct_nwaves;
    out->direct_unroll = row->direct_unroll;
    if (ctx->nranks == 2 && out->proto == AR_PROTO_LL) {
        // With two ranks the peer-direct Simple ring waits for no flag at
        // all (its one reduction hop is a peer read, its one all-gather hop
        // waits for nothing), so the LL rows defer to the default there.
        out->proto = AR_PROTO_AUTO;
        out->nchannels = 0;
        out->chunk_bytes = 0;
        out->nwaves = 0;
    }
    return 0;
}

int ar_set_tuner(ar_tuner_fn fn, void *user) { return install(fn, user, false, nullptr); }

int ar_reload_tuner(ar_tuner_fn fn, void *user, ar_reload_stats *stats)
{
    return install(fn, user, true, stats);
}

int ar_tune(const ar_tune_ctx *ctx, ar_tune_out *out)
{
    if (!ctx || !out) return AR_ERR_ARG;
    if (ctx->nranks < 1 || ctx->nranks > AR_MAX_RANKS) return AR_ERR_ARG;
    if (ctx->dtype != AR_FLOAT32 && ctx->dtype != AR_BFLOAT16) return AR_ERR_ARG;
    const int max_ch = clamp_int(ctx->max_channels > 0 ? ctx->max_channels : AR_MAX_CHANNELS, 1,
                                 AR_MAX_CHANNELS);
    TunerSlot *slot = pin_active();
    ar_tune_out t = {AR_PROTO_AUTO, 0, 0, 0, AR_ALGO_AUTO, 0, 0};
    int rc = slot->fn(ctx, &t, slot->user);
    unpin(slot);

    // No opinion on the protocol means the fixed default's ring choice.
    if (rc == 0 && t.proto == AR_PROTO_AUTO && valid_algo(t.algo)) {
        t.proto = kDefaultProto;
        t.nchannels = t.nchannels > 0 ? t.nchannels : kDefaultChannels;
    }
    bool fallback = rc != 0 || !valid_proto(t.proto) || !valid_algo(t.algo) || t.nchannels < 0 || t.nwaves < 0 ||
                    t.direct_parts < 0 || t.direct_nwaves < 0 || t.direct_unroll < 0 || t.direct_unroll > 2;
    if (fallback) {
        t.proto = kDefaultProto;
        t.nchannels = kDefaultChannels;
        t.chunk_bytes = 0;
        t.nwaves = 0;
        t.algo = AR_ALGO_RING;
        t.direct_parts = 0;
        t.direct_nwaves = 0;
        t.direct_unroll = 0;
    }
    if (t.direct_nwaves > AR_MAX_WAVES) t.direct_nwaves = AR_MAX_WAVES;
    if (t.algo == AR_ALGO_AUTO) t.algo = AR_ALGO_RING;
    if (t.nchannels == 0) t.nchannels = kDefaultChannels;
    t.nchannels = clamp_int(t.nchannels, 1, max_ch);
    t.chunk_bytes = t.chunk_bytes ? clamp_chunk(t.chunk_bytes) : default_chunk_bytes(t.proto);
    t.nwaves = t.nwaves ? clamp_int(t.nwaves, 1, AR_MAX_WAVES) : default_nwaves(t.proto);
    *out = t;
    return AR_OK;
}

int ar_plan_geometry(const ar_plan_desc *desc, ar_plan_info *out)
{
    if (!desc || !out) return AR_ERR_ARG;
    int maxc = desc->max_channels > 0 ? desc->max_channels : AR_MAX_CHANNELS;
    return resolve_geometry(desc, maxc, out);
}

const char *ar_strerror(int code)
{
    switch (code) {
    case AR_OK: return "success";
    case AR_ERR_ARG: return "invalid argument";
    case AR_ERR_UNSUPPORTED: return "unsupported request";
    case AR_ERR_NOMEM: return "out of memory";
    case AR_ERR_HIP: return "HIP runtime error";
    case AR_ERR_OCCUPANCY: return "grid cannot be co-resident on the device";
    case AR_ERR_TIMEOUT: return "flag wait exceeded the watchdog";
    case AR_ERR_STATE: return "plan is in an error state";
    case AR_ERR_SCRATCH: return "request needs more than the static scratch of the allocation-free call";
    default: return "unknown error";
    }
}

int ar_last_error(void) { return g_last_error; }

int ar_version(void) { return AR_VERSION; }

}  // extern "C"
