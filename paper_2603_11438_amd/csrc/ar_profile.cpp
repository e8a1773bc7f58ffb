// Telemetry shared by the profiler hook and the tuner, and the adaptive
// channel-count tuner that reads it: host-only C++ with no HIP dependency.
//
// Paper section 3.3 (Listing 1, profiler-to-tuner closed loop): a profiler
// program writes the latest latency and channel count of a communicator
// into a shared typed map; the tuner looks the entry up (a lookup can find
// nothing and must be checked) and chooses the channel count from it.
// Paper section 5.3 (composability): an adaptive policy starts at 2
// channels, ramps to 12 while latency samples arrive, drops back to 2 under
// a 10x latency spike, and ramps up again after the spike.
//
// The map is a fixed-size open-addressing table (like an eBPF hash map of
// fixed capacity).  Every field a thread may read while another writes is a
// 64-bit atomic, and the latency and the channel count it was measured at
// are packed into one word, so a reader never sees a latency paired with
// the wrong channel count.
#include <atomic>
#include <stddef.h>
#include <stdint.h>

#include "ar.h"
#include "ar_internal.h"

namespace ar {
namespace {

constexpr int kCapacity = 1024;
constexpr int kMaxTrackedChannels = 64;  // per-channel-count baselines kept for 1..64
constexpr uint64_t kLatBits = 48;
constexpr uint64_t kLatMask = (1ull << kLatBits) - 1;

struct Entry {
    std::atomic<uint64_t> key{0};      // comm_id + 1; 0 = empty
    std::atomic<uint64_t> sample{0};   // latency_ns (low 48 bits) | channels << 48
    std::atomic<uint64_t> samples{0};  // number of samples recorded
    // Adaptive-tuner state (written by the tuner only).
    std::atomic<uint64_t> decision{0};  // channels (low 16) | calls since last change << 16
    std::atomic<uint64_t> baseline[kMaxTrackedChannels + 1];  // fastest latency seen per channel count
};

Entry g_map[kCapacity];

uint64_t mix(uint64_t x)
{
    x ^= x >> 33;
    x *= 0xff51afd7ed558ccdull;
    x ^= x >> 33;
    return x;
}

// Find the entry of comm_id; insert it if `create`.  Returns nullptr when
// absent (and not created) or when the table is full.
Entry *find(uint64_t comm_id, bool create)
{
    const uint64_t key = comm_id + 1;
    if (key == 0) return nullptr;  // comm_id UINT64_MAX is not storable
    uint64_t h = mix(comm_id) % kCapacity;
    for (int i = 0; i < kCapacity; ++i) {
        Entry &e = g_map[(h + i) % kCapacity];
        uint64_t k = e.key.load(std::memory_order_acquire);
        if (k == key) return &e;
        if (k == 0) {
            if (!create) return nullptr;
            uint64_t expected = 0;
            if (e.key.compare_exchange_strong(expected, key, std::memory_order_acq_rel)) return &e;
            if (expected == key) return &e;
        }
    }
    return nullptr;
}

}  // namespace
}  // namespace ar

using namespace ar;

extern "C" {

int ar_profile_record(uint64_t comm_id, uint64_t latency_ns, int nchannels)
{
    if (nchannels < 0 || nchannels > 0xFFFF) return AR_ERR_ARG;
    Entry *e = find(comm_id, true);
    if (!e) return AR_ERR_NOMEM;
    if (latency_ns > kLatMask) latency_ns = kLatMask;
    e->sample.store(latency_ns | ((uint64_t)nchannels << kLatBits), std::memory_order_release);
    e->samples.fetch_add(1, std::memory_order_acq_rel);
    return AR_OK;
}

int ar_profile_lookup(uint64_t comm_id, ar_latency_state *out)
{
    if (!out) return AR_ERR_ARG;
    Entry *e = find(comm_id, false);
    if (!e || e->samples.load(std::memory_order_acquire) == 0) return AR_ERR_ARG;
    uint64_t s = e->sample.load(std::memory_order_acquire);
    out->comm_id = comm_id;
    out->latency_ns = s & kLatMask;
    out->nchannels = (int)(s >> kLatBits);
    out->samples = e->samples.load(std::memory_order_acquire);
    return AR_OK;
}

void ar_profile_clear(void)
{
    for (Entry &e : g_map) {
        e.sample.store(0, std::memory_order_relaxed);
        e.samples.store(0, std::memory_order_relaxed);
        e.decision.store(0, std::memory_order_relaxed);
        for (auto &b : e.baseline) b.store(0, std::memory_order_relaxed);
        e.key.store(0, std::memory_order_release);
    }
}

// Adaptive channels (see the file comment).  The rule, per decision for
// ctx->comm_id:
//   * no telemetry for the communicator yet: min_channels;
//   * the latest sample ran at c channels with latency L.  The reference is
//     the fastest latency ever seen at c or fewer channels (adding channels
//     should not make a run slower, so this also covers a channel count
//     that has no history yet); if L exceeds backoff_ratio x the reference,
//     the link is contended: drop to min_channels;
//   * otherwise count the decision, and after ramp_calls decisions without
//     contention add one channel, up to max_channels.
int ar_tuner_adaptive(const ar_tune_ctx *ctx, ar_tune_out *out, void *user)
{
    if (!ctx || !out) return -1;
    ar_adaptive_cfg cfg = {2, 12, 9000, 4, AR_PROTO_SIMPLE};
    if (user) cfg = *static_cast<const ar_adaptive_cfg *>(user);
    if (cfg.min_channels < 1 || cfg.max_channels < cfg.min_channels || cfg.ramp_calls == 0 || cfg.backoff_ratio < 1)
        return -1;
    out->proto = cfg.proto;
    out->chunk_bytes = 0;
    out->nwaves = 0;
    out->algo = AR_ALGO_RING;
    out->direct_parts = 0;
    out->direct_nwaves = 0;
    out->direct_unroll = 0;
    Entry *e = find(ctx->comm_id, false);
    if (!e || e->samples.load(std::memory_order_acquire) == 0) {
        out->nchannels = cfg.min_channels;
        return 0;
    }
    const uint64_t s = e->sample.load(std::memory_order_acquire);
    const uint64_t lat = s & kLatMask;
    const int sch = (int)(s >> kLatBits);
    bool contended = false;
    if (sch >= 1 && sch <= kMaxTrackedChannels) {
        std::atomic<uint64_t> &b = e->baseline[sch];
        uint64_t base = b.load(std::memory_order_acquire);
        while ((base == 0 || lat < base) && !b.compare_exchange_weak(base, lat, std::memory_order_acq_rel)) {
        }
        uint64_t ref = lat;
        for (int c = 1; c <= sch; ++c) {
            uint64_t v = e->baseline[c].load(std::memory_order_acquire);
            if (v != 0 && v < ref) ref = v;
        }
        contended = lat > (uint64_t)cfg.backoff_ratio * ref;
    }
    uint64_t d = e->decision.load(std::memory_order_acquire);
    uint64_t nd;
    do {
        int ch = (int)(d & 0xFFFF);
        uint64_t calls = d >> 16;
        if (ch < cfg.min_channels || ch > cfg.max_channels) ch = cfg.min_channels;
        if (contended) {
            ch = cfg.min_channels;
            calls = 0;
        } else if (++calls >= cfg.ramp_calls) {
            if (ch < cfg.max_channels) ++ch;
            calls = 0;
        }
        nd = (uint64_t)ch | (calls << 16);
    } while (!e->decision.compare_exchange_weak(d, nd, std::memory_order_acq_rel));
    out->nchannels = (int)(nd & 0xFFFF);
    return 0;
}

// The closed-loop tuner of the paper's Listing 1 (section 3.3), with its
// tree choice mapped to this library's small-message algorithm (direct):
//   * no telemetry entry for the communicator: 4 channels and nothing else
//     (algorithm and protocol stay without an opinion, so the library's
//     default applies);
//   * otherwise messages of at most 32 KiB use the small-message algorithm,
//     larger ones the ring, with the Simple protocol, and when the last
//     recorded latency exceeds 1 ms, one channel more than that run had (at
//     most 16), otherwise the same count.
int ar_tuner_size_adaptive(const ar_tune_ctx *ctx, ar_tune_out *out, void *user)
{
    (void)user;
    if (!ctx || !out) return -1;
    Entry *e = find(ctx->comm_id, false);
    if (!e || e->samples.load(std::memory_order_acquire) == 0) {
        out->nchannels = 4;
        return 0;
    }
    out->proto = AR_PROTO_SIMPLE;
    out->chunk_bytes = 0;
    out->nwaves = 0;
    out->direct_parts = 0;
    out->direct_nwaves = 0;
    out->direct_unroll = 0;
    out->algo = ctx->msg_bytes <= 32u * 1024u ? AR_ALGO_DIRECT : AR_ALGO_RING;
    const uint64_t s = e->sample.load(std::memory_order_acquire);
    const uint64_t lat = s & kLatMask;
    int ch = (int)(s >> kLatBits);
    if (ch < 1) ch = 1;
    if (lat > 1000000u) ch = ch + 1 < 16 ? ch + 1 : 16;
    out->nchannels = ch;
    return 0;
}

}  // extern "C"
