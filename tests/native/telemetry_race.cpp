// Concurrent profiler records, lookups and adaptive-tuner decisions on the
// shared telemetry map, run under ThreadSanitizer by
// tests/test_closed_loop.py.  Every lookup must return a sample whose
// latency and channel count were recorded together (writers record
// latency = 1000 * channels).
#include <atomic>
#include <cstdio>
#include <thread>
#include <vector>

#include "ar.h"

int main()
{
    ar_profile_clear();
    if (ar_set_tuner(ar_tuner_adaptive, nullptr) != AR_OK) return 2;
    std::atomic<long> torn{0}, bad{0};
    std::vector<std::thread> th;
    for (int t = 0; t < 3; ++t)
        th.emplace_back([&, t] {
            for (int i = 0; i < 20000; ++i) {
                int ch = 1 + (i + t) % 16;
                if (ar_profile_record((uint64_t)(i % 8), 1000ull * ch, ch) != AR_OK) bad.fetch_add(1);
            }
        });
    for (int t = 0; t < 3; ++t)
        th.emplace_back([&, t] {
            for (int i = 0; i < 20000; ++i) {
                ar_latency_state s;
                if (ar_profile_lookup((uint64_t)((i + t) % 8), &s) == AR_OK && s.latency_ns != 1000ull * s.nchannels)
                    torn.fetch_add(1);
                ar_tune_ctx c = {AR_COLL_ALLREDUCE, 1u << 20, 8, AR_FLOAT32, 64, (uint64_t)(i % 8)};
                ar_tune_out o;
                if (ar_tune(&c, &o) != AR_OK || o.nchannels < 2 || o.nchannels > 12) bad.fetch_add(1);
            }
        });
    for (auto &x : th) x.join();
    ar_set_tuner(nullptr, nullptr);
    printf("torn %ld bad %ld\n", torn.load(), bad.load());
    return torn.load() == 0 && bad.load() == 0 ? 0 : 1;
}
