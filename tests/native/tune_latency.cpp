// Host decision latency of ar_tune (context for the paper's per-decision
// costs, section 5.1 Table 1): 1,000,000 decisions of the built-in table
// for message sizes cycling through 4 KiB .. 128 MiB, each timed on its own
// with steady_clock; the cost of an empty timed interval is measured the
// same way and reported beside it.  Prints P50 / P99 in nanoseconds.
#include <algorithm>
#include <chrono>
#include <cstdio>
#include <vector>

#include "ar.h"

static long pct(std::vector<long> &v, double p)
{
    std::sort(v.begin(), v.end());
    return v[(size_t)(p * (v.size() - 1))];
}

int main(int argc, char **argv)
{
    const int n = argc > 1 ? atoi(argv[1]) : 1000000;
    using clk = std::chrono::steady_clock;
    std::vector<long> t(n), e(n);
    ar_tune_out o;
    volatile int sink = 0;
    for (int i = 0; i < n; ++i) {
        ar_tune_ctx c = {AR_COLL_ALLREDUCE, (size_t)4096 << (i % 16), 8, AR_FLOAT32, 64, 0};
        auto a = clk::now();
        ar_tune(&c, &o);
        auto b = clk::now();
        t[i] = (long)std::chrono::duration_cast<std::chrono::nanoseconds>(b - a).count();
        sink += o.nchannels;
    }
    for (int i = 0; i < n; ++i) {
        auto a = clk::now();
        auto b = clk::now();
        e[i] = (long)std::chrono::duration_cast<std::chrono::nanoseconds>(b - a).count();
    }
    printf("ar_tune ns p50 %ld p99 %ld | empty interval ns p50 %ld p99 %ld | n %d\n", pct(t, 0.5), pct(t, 0.99),
           pct(e, 0.5), pct(e, 0.99), n);
    return sink < 0;
}
