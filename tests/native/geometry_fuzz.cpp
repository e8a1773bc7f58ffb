// Randomised plan-geometry and tuner checks, built from the host-only tuner
// source with g++ under AddressSanitizer and UndefinedBehaviorSanitizer and
// run by tests/test_tuner_reload.py.  For random descriptors (valid and
// invalid) ar_plan_geometry must either reject them or return a geometry
// whose segments, channel sub-ranges, chunks and FIFO slots cover the
// buffer; ar_tune must always return a complete, in-range decision.
#include <cstdio>
#include <cstdint>
#include <random>

#include "ar.h"

int main(int argc, char **argv)
{
    const int iters = argc > 1 ? atoi(argv[1]) : 200000;
    std::mt19937_64 rng(11438);
    long accepted = 0, failures = 0;
    for (int i = 0; i < iters; ++i) {
        ar_plan_desc d = {};
        d.nranks = (int)(rng() % 20) - 1;
        d.dtype = (int)(rng() % 3);
        int lg = (int)(rng() % 36);
        d.count = (size_t)(rng() % ((1ull << lg) + 1));
        d.proto = (int)(rng() % 5) - 1;
        d.nchannels = (int)(rng() % 300) - 2;
        d.chunk_bytes = (rng() % 4) ? (size_t)(rng() % (80u << 20)) : 0;
        d.fifo_depth = (int)(rng() % 20) - 1;
        d.nwaves = (int)(rng() % 20) - 1;
        d.placement = (int)(rng() % 3);
        d.max_channels = (int)(rng() % 300);
        d.algo = (int)(rng() % 4);
        ar_plan_info g;
        int rc = ar_plan_geometry(&d, &g);
        if (rc != AR_OK) continue;
        ++accepted;
        const uint64_t e = g.dtype == AR_FLOAT32 ? 4 : 2, A = 16 / e, N = (uint64_t)g.nranks;
        bool ok = g.seg_elems * N >= g.count && g.seg_elems % A == 0;
        if (g.grid > 0 && g.algo == AR_ALGO_DIRECT) {
            ok = ok && g.grid == g.nchannels * g.nranks && g.block == 64 * g.nwaves && g.nchannels >= 1;
            ok = ok && g.chan_elems * (uint64_t)g.nchannels >= g.seg_elems && g.chan_elems % A == 0;
            ok = ok && g.fifo_bytes == 0 && g.msgs_per_run == 0 && g.nwaves >= 1 && g.nwaves <= AR_MAX_WAVES;
        } else if (g.grid > 0) {
            ok = ok && g.algo == AR_ALGO_RING;
            ok = ok && g.grid == g.nchannels * g.nranks && g.block == 64 * g.nwaves;
            ok = ok && g.chan_elems * (uint64_t)g.nchannels >= g.seg_elems && g.chan_elems % A == 0;
            ok = ok && g.chunk_elems >= A && g.chunk_elems <= g.chan_elems && g.chunk_elems % A == 0;
            ok = ok && g.nchunks * g.chunk_elems >= g.chan_elems;
            ok = ok && g.wave_elems * (uint64_t)g.nwaves >= g.chunk_elems;
            // a ring plan without AR_PLAN_FIFO_ONLY starts each chain with a peer read
            ok = ok && g.msgs_per_run == g.nchunks * (2 * N - 2 - (uint64_t)g.peer_direct);
            ok = ok && g.peer_direct == 1;
            ok = ok && g.slot_bytes % 256 == 0 && g.slot_bytes >= g.wave_elems * 4;
            ok = ok && g.fifo_bytes == (uint64_t)g.nchannels * N * g.nwaves * g.fifo_depth * g.slot_bytes;
            ok = ok && g.fifo_depth >= 2 && g.fifo_depth <= 16 && g.nwaves >= 1 && g.nwaves <= AR_MAX_WAVES;
        }
        if (!ok) {
            ++failures;
            if (failures < 5) fprintf(stderr, "bad geometry at iter %d\n", i);
        }
        ar_tune_ctx c = {AR_COLL_ALLREDUCE, (size_t)d.count * 4, g.nranks, g.dtype, d.max_channels, 0};
        ar_tune_out o;
        if (ar_tune(&c, &o) != AR_OK || (o.proto != AR_PROTO_LL && o.proto != AR_PROTO_LL128 &&
                                         o.proto != AR_PROTO_SIMPLE) ||
            o.nchannels < 1 || o.nwaves < 1 || o.chunk_bytes < 16 ||
            (o.algo != AR_ALGO_RING && o.algo != AR_ALGO_DIRECT) || o.direct_parts < 0 || o.direct_nwaves < 0)
            ++failures;
    }
    printf("iters %d accepted %ld failures %ld\n", iters, accepted, failures);
    return failures == 0 && accepted > iters / 50 ? 0 : 1;
}
