// Concurrency test of the tuner hot reload (ar_set_tuner / ar_reload_tuner /
// ar_tune), built from the host-only tuner source with g++ under a
// sanitizer and run by tests/test_tuner_reload.py.
//
// Reader threads make decisions continuously while a writer thread keeps
// swapping between freshly created tuner instances.  Each instance answers
// a decision that encodes its own identity in every output field, so a
// decision mixing two instances ("torn") is detectable.  Checked:
//   * every call returns AR_OK with a complete decision (no lost calls);
//   * no torn decision;
//   * after a reload returns, the replaced instance is never called again
//     (the drain guarantee);
//   * a malformed candidate is rejected and the current tuner keeps serving.
// Prints "swap_ns p50 p99 max" and "calls N".
#include <atomic>
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <thread>
#include <vector>

#include "ar.h"

namespace {

struct Instance {
    int id;
    std::atomic<long> calls{0};
    std::atomic<bool> retired{false};
    std::atomic<long> calls_after_retire{0};
};

int instance_tuner(const ar_tune_ctx *ctx, ar_tune_out *out, void *user)
{
    Instance *in = static_cast<Instance *>(user);
    in->calls.fetch_add(1, std::memory_order_relaxed);
    if (in->retired.load(std::memory_order_acquire)) in->calls_after_retire.fetch_add(1);
    // Every field carries the instance id.
    const int k = in->id % 3;
    out->proto = k == 0 ? AR_PROTO_LL : (k == 1 ? AR_PROTO_LL128 : AR_PROTO_SIMPLE);
    out->nchannels = 1 + in->id % 50;
    out->chunk_bytes = 4096u * (size_t)(1 + in->id % 97);
    out->nwaves = 1 + in->id % 16;
    out->algo = AR_ALGO_RING;
    out->direct_parts = 0;
    out->direct_nwaves = 0;
    (void)ctx;
    return 0;
}

int malformed_tuner(const ar_tune_ctx *ctx, ar_tune_out *out, void *)
{
    out->proto = ctx->msg_bytes > (64u << 20) ? 9 : AR_PROTO_SIMPLE;  // bad only for big messages
    out->nchannels = 4;
    out->chunk_bytes = 0;
    out->nwaves = 0;
    out->algo = AR_ALGO_RING;
    out->direct_parts = 0;
    out->direct_nwaves = 0;
    return 0;
}

bool consistent(const ar_tune_out &o)
{
    // Recover the id from nchannels and nwaves; every other field must agree.
    for (int id = 0; id < 4000; ++id) {
        int k = id % 3;
        int proto = k == 0 ? AR_PROTO_LL : (k == 1 ? AR_PROTO_LL128 : AR_PROTO_SIMPLE);
        if (o.proto == proto && o.nchannels == 1 + id % 50 && o.chunk_bytes == 4096u * (size_t)(1 + id % 97) &&
            o.nwaves == 1 + id % 16)
            return true;
    }
    return false;
}

}  // namespace

int main(int argc, char **argv)
{
    const long total_calls = argc > 1 ? atol(argv[1]) : 400000;
    const int nreaders = argc > 2 ? atoi(argv[2]) : 4;
    std::vector<Instance *> instances;
    instances.reserve(4000);
    auto make = [&](int id) {
        Instance *in = new Instance();
        in->id = id;
        instances.push_back(in);
        return in;
    };
    Instance *cur = make(0);
    if (ar_set_tuner(instance_tuner, cur) != AR_OK) return 2;

    std::atomic<long> done{0}, bad{0}, torn{0};
    std::atomic<bool> stop{false};
    std::vector<std::thread> readers;
    for (int t = 0; t < nreaders; ++t) {
        readers.emplace_back([&, t] {
            long mine = total_calls / nreaders;
            ar_tune_ctx c = {AR_COLL_ALLREDUCE, (size_t)4096 << (t % 16), 8, AR_FLOAT32, AR_MAX_CHANNELS, (uint64_t)t};
            for (long i = 0; i < mine; ++i) {
                ar_tune_out o = {-7, -7, 7, -7, -7, -7, -7};
                int rc = ar_tune(&c, &o);
                if (rc != AR_OK) bad.fetch_add(1);
                else if (!consistent(o)) torn.fetch_add(1);
                done.fetch_add(1, std::memory_order_relaxed);
            }
        });
    }
    std::vector<long> swap_ns;
    int next_id = 1, rejected = 0, rejected_ok = 0;
    while (done.load() < total_calls - total_calls / 50 && next_id < 3900) {
        if (next_id % 7 == 0) {
            ar_reload_stats st;
            int rc = ar_reload_tuner(malformed_tuner, nullptr, &st);
            ++rejected;
            if (rc == AR_ERR_ARG) ++rejected_ok;
            // the current instance must still be the one answering
            ar_tune_ctx c = {AR_COLL_ALLREDUCE, 1u << 20, 8, AR_FLOAT32, AR_MAX_CHANNELS, 0};
            ar_tune_out o;
            ar_tune(&c, &o);
            if (o.nchannels != 1 + cur->id % 50) bad.fetch_add(1);
        }
        Instance *nx = make(next_id++);
        ar_reload_stats st;
        if (ar_reload_tuner(instance_tuner, nx, &st) != AR_OK) return 3;
        swap_ns.push_back((long)st.swap_ns);
        // drained: the replaced instance must never run again
        cur->retired.store(true, std::memory_order_release);
        cur = nx;
        std::this_thread::sleep_for(std::chrono::microseconds(50));
    }
    for (auto &r : readers) r.join();
    long after = 0;
    for (Instance *in : instances) after += in->calls_after_retire.load();
    std::sort(swap_ns.begin(), swap_ns.end());
    auto pct = [&](double p) { return swap_ns.empty() ? 0L : swap_ns[(size_t)(p * (swap_ns.size() - 1))]; };
    printf("calls %ld bad %ld torn %ld after_retire %ld reloads %zu rejected %d/%d\n", done.load(), bad.load(),
           torn.load(), after, swap_ns.size(), rejected_ok, rejected);
    printf("swap_ns p50 %ld p99 %ld max %ld\n", pct(0.5), pct(0.99), pct(1.0));
    ar_set_tuner(nullptr, nullptr);
    const bool ok = bad.load() == 0 && torn.load() == 0 && after == 0 && rejected_ok == rejected &&
                    done.load() == (total_calls / nreaders) * nreaders && !swap_ns.empty();
    return ok ? 0 : 1;
}
