// Host-only test of the ring launch gate (ring_gate.h) with a fake stream
// API that keeps a log of device waits, event waits and records.  Checks:
//   * while a device has seen one stream, launches cost nothing (no event);
//   * the first launch on a second stream waits for the whole device once
//     and switches the device to ordered mode;
//   * in ordered mode the event is recorded after every launch, and a launch
//     on another stream than the last waits for the event of that launch;
//   * launches being captured are neither ordered nor recorded;
//   * devices keep separate state; out-of-range devices are refused;
//   * an API error stops the launch sequence and is returned;
//   * under concurrent launchers (run with ThreadSanitizer) no two launches
//     on different streams overlap: replayed, the log shows every stream
//     switch behind a device wait or a wait for the previous launch.
#include <stdio.h>
#include <stdlib.h>

#include <atomic>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "ring_gate.h"

namespace {

struct Op {
    char kind;    // 'w' wait, 'r' record, 'c' create, 'S' device wait, 'L' launch
    int stream;
    int event;    // event id; for 'r' the generation recorded, for 'w' the generation awaited
    int dev;
};

std::mutex g_log_mu;
std::vector<Op> g_log;
std::atomic<int> g_fail_next{0};  // make the next API call of this kind fail: 'w' or 'r'
std::atomic<int> g_capturing_stream{-1};
int g_event_gen[16];  // generation of each event (bumped by every record)

void log_op(Op o)
{
    std::lock_guard<std::mutex> g(g_log_mu);
    g_log.push_back(o);
}

struct FakeApi {
    using Stream = int;
    using Event = int;
    static int capturing(Stream s, bool *yes)
    {
        *yes = s == g_capturing_stream.load();
        return 0;
    }
    static int sync_device()
    {
        log_op({'S', -1, -1, -1});
        return 0;
    }
    static int create(Event *e)
    {
        static std::atomic<int> next{0};
        *e = next.fetch_add(1);
        log_op({'c', -1, *e, -1});
        return 0;
    }
    static int wait(Stream s, Event e)
    {
        if (g_fail_next.load() == 'w') {
            g_fail_next = 0;
            return 7;
        }
        log_op({'w', s, g_event_gen[e], -1});
        return 0;
    }
    static int record(Event e, Stream s)
    {
        if (g_fail_next.load() == 'r') {
            g_fail_next = 0;
            return 9;
        }
        ++g_event_gen[e];
        log_op({'r', s, g_event_gen[e], -1});
        return 0;
    }
};

int failures = 0;
#define CHECK(c)                                                              \
    do {                                                                      \
        if (!(c)) {                                                           \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #c); \
            ++failures;                                                       \
        }                                                                     \
    } while (0)

using Gate = ar::RingGate<FakeApi, 4>;

// One launch through the gate; returns the gate's code.
int launch(Gate &g, int dev, int stream)
{
    Gate::Ticket t;
    int rc = g.before(dev, stream, t);
    if (rc != 0) return rc;
    log_op({'L', stream, -1, dev});
    return g.after(t);
}

std::vector<Op> take_log()
{
    std::lock_guard<std::mutex> g(g_log_mu);
    std::vector<Op> v;
    v.swap(g_log);
    return v;
}

std::string kinds(const std::vector<Op> &v)
{
    std::string s;
    for (const Op &o : v) s += o.kind;
    return s;
}

void test_sequences()
{
    Gate g;
    // one stream: nothing but the launches
    CHECK(launch(g, 0, 1) == 0);
    CHECK(kinds(take_log()) == "L");
    CHECK(launch(g, 0, 1) == 0);
    CHECK(kinds(take_log()) == "L");
    CHECK(!g.ordered(0));
    // a second stream: one device wait, then ordered mode (record after)
    CHECK(launch(g, 0, 2) == 0);
    CHECK(kinds(take_log()) == "cSLr");
    CHECK(g.ordered(0));
    int last = -1;
    CHECK(g.last_stream(0, &last) && last == 2);
    // same stream in ordered mode: no wait, record after
    CHECK(launch(g, 0, 2) == 0);
    CHECK(kinds(take_log()) == "Lr");
    // back to stream 1: wait for stream 2's last launch (generation 2)
    CHECK(launch(g, 0, 1) == 0);
    auto v = take_log();
    CHECK(kinds(v) == "wLr");
    CHECK(v[0].stream == 1 && v[0].event == 2);

    // a capturing stream is neither ordered nor recorded, and does not
    // change which launch the next one waits for
    g_capturing_stream = 5;
    CHECK(launch(g, 0, 5) == 0);
    CHECK(kinds(take_log()) == "L");
    g_capturing_stream = -1;
    CHECK(g.last_stream(0, &last) && last == 1);
    CHECK(launch(g, 0, 1) == 0);
    CHECK(kinds(take_log()) == "Lr");

    // device 1 has its own state: one stream costs nothing there
    CHECK(launch(g, 1, 2) == 0);
    CHECK(kinds(take_log()) == "L");
    CHECK(launch(g, 1, 2) == 0);
    CHECK(kinds(take_log()) == "L");
    CHECK(!g.ordered(1));

    // out-of-range devices are refused before anything happens
    Gate::Ticket t;
    CHECK(g.before(4, 1, t) != 0);
    CHECK(g.before(-1, 1, t) != 0);
    CHECK(take_log().empty());

    // a failing wait stops the launch and is returned
    g_fail_next = 'w';
    CHECK(launch(g, 0, 3) == 7);
    CHECK(kinds(take_log()).empty());
    // a failing record is returned after the launch
    g_fail_next = 'r';
    CHECK(launch(g, 0, 3) == 9);
    CHECK(kinds(take_log()) == "wL");
}

// Concurrent launchers on several streams of one device.  Replaying the log
// in order: before the device wait every launch is on one stream; after it,
// each launch on a stream other than the previous launch's is preceded
// (after that previous launch's record) by a wait on its stream for the
// generation the previous launch recorded.
void test_concurrent()
{
    Gate g;
    take_log();
    const int kThreads = 6, kLaunches = 3000;
    std::vector<std::thread> th;
    for (int i = 0; i < kThreads; ++i)
        th.emplace_back([&g, i] {
            for (int k = 0; k < kLaunches; ++k) {
                const int stream = 10 + (i + k) % 3;  // threads share streams
                if (launch(g, 2, stream) != 0) abort();
            }
        });
    for (auto &t : th) t.join();
    auto v = take_log();
    bool ordered = false;
    int syncs = 0, first_stream = -1;
    int prev_stream = -1, prev_gen = 0, pending_wait_gen = -1, pending_wait_stream = -1;
    int launches = 0, waits = 0;
    for (size_t i = 0; i < v.size(); ++i) {
        const Op &o = v[i];
        if (o.kind == 'S') {
            ++syncs;
            ordered = true;
        } else if (o.kind == 'w') {
            pending_wait_gen = o.event;
            pending_wait_stream = o.stream;
            ++waits;
        } else if (o.kind == 'L') {
            if (!ordered) {
                if (first_stream < 0) first_stream = o.stream;
                CHECK(o.stream == first_stream);
            } else if (prev_stream >= 0 && o.stream != prev_stream) {
                CHECK(pending_wait_stream == o.stream && pending_wait_gen == prev_gen);
            } else {
                CHECK(pending_wait_gen == -1);
            }
            pending_wait_gen = pending_wait_stream = -1;
            ++launches;
        } else if (o.kind == 'r') {
            // the record right after a launch marks that launch
            CHECK(i > 0 && v[i - 1].kind == 'L' && v[i - 1].stream == o.stream);
            prev_stream = o.stream;
            prev_gen = o.event;
        }
    }
    CHECK(syncs == 1);
    CHECK(launches == kThreads * kLaunches);
    CHECK(waits > 0);
    printf("concurrent: %d launches, %d waits, %d device wait\n", launches, waits, syncs);
}

}  // namespace

int main()
{
    test_sequences();
    test_concurrent();
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("ring gate: ok\n");
    return 0;
}
