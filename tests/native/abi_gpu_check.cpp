// libar through its C ABI alone (no Python, no torch): eight rank buffers
// from hipMalloc, AllReduces planned with ar_plan and ar_plan_ex (the
// tuner's choice, the LL ring, LL128 and Simple rings, the direct
// algorithm, in place and out of place, fp32 and bf16), each checked on the
// host against exact integer sums.  Prints one line per case and "abi gpu
// check: ok" at the end; exits non-zero on the first failure.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "ar.h"

namespace {

const int N = 8;
const size_t COUNT = 100003;  // not a multiple of N times a 16-byte unit

bool hip_ok(hipError_t e, const char *what)
{
    if (e == hipSuccess) return true;
    std::printf("%s: %s\n", what, hipGetErrorString(e));
    return false;
}

// Rank r's element i: a small integer, so every partial sum is exact in
// fp32 and every value and sum is exact in bf16.
float value(int r, size_t i) { return (float)((int)((i * 7 + (size_t)r * 13) % 33) - 16); }

uint16_t to_bf16(float f)
{
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);  // exact: the values have at most 8 significant bits
}

float from_bf16(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

struct Case {
    const char *name;
    bool ex;     // ar_plan_ex with the fields below, else ar_plan(proto, nchannels)
    int dtype, proto, nchannels, algo;
    bool oop;
};

bool run_case(const Case &c)
{
    const size_t esz = c.dtype == AR_FLOAT32 ? 4 : 2;
    std::vector<void *> in(N, nullptr), out(N, nullptr);
    std::vector<float> want(COUNT, 0.0f);
    for (int r = 0; r < N; ++r)
        for (size_t i = 0; i < COUNT; ++i) want[i] += value(r, i);
    bool ok = true;
    for (int r = 0; r < N && ok; ++r) {
        ok = hip_ok(hipMalloc(&in[r], COUNT * esz), "hipMalloc") &&
             hip_ok(hipMalloc(&out[r], COUNT * esz), "hipMalloc");
        if (!ok) break;
        std::vector<uint8_t> h(COUNT * esz);
        for (size_t i = 0; i < COUNT; ++i) {
            if (c.dtype == AR_FLOAT32) {
                const float v = value(r, i);
                std::memcpy(&h[i * 4], &v, 4);
            } else {
                const uint16_t v = to_bf16(value(r, i));
                std::memcpy(&h[i * 2], &v, 2);
            }
        }
        ok = hip_ok(hipMemcpy(in[r], h.data(), h.size(), hipMemcpyHostToDevice), "hipMemcpy");
    }
    ar_plan_t *p = nullptr;
    if (ok) {
        if (c.ex) {
            ar_plan_desc d;
            std::memset(&d, 0, sizeof d);
            d.nranks = N;
            d.count = COUNT;
            d.dtype = c.dtype;
            d.proto = c.proto;
            d.nchannels = c.nchannels;
            d.algo = c.algo;
            p = ar_plan_ex(&d);
        } else {
            p = ar_plan(N, COUNT, c.dtype, c.proto, c.nchannels);
        }
        if (!p) {
            std::printf("%s: plan: %s\n", c.name, ar_strerror(ar_last_error()));
            ok = false;
        }
    }
    if (ok) {
        const int rc = c.oop ? ar_run_oop(p, in.data(), out.data(), nullptr) : ar_run(p, in.data(), nullptr);
        ok = rc == AR_OK && hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
        if (rc != AR_OK) std::printf("%s: run: %s\n", c.name, ar_strerror(rc));
        if (ok && ar_plan_status(p) != AR_OK) {
            std::printf("%s: plan status %s\n", c.name, ar_strerror(ar_plan_status(p)));
            ok = false;
        }
    }
    for (int r = 0; r < N && ok; ++r) {
        std::vector<uint8_t> h(COUNT * esz);
        ok = hip_ok(hipMemcpy(h.data(), c.oop ? out[r] : in[r], h.size(), hipMemcpyDeviceToHost), "hipMemcpy");
        for (size_t i = 0; i < COUNT && ok; ++i) {
            float got;
            if (c.dtype == AR_FLOAT32) {
                std::memcpy(&got, &h[i * 4], 4);
            } else {
                uint16_t g;
                std::memcpy(&g, &h[i * 2], 2);
                got = from_bf16(g);
            }
            if (got != want[i]) {
                std::printf("%s: rank %d element %zu is %g, want %g\n", c.name, r, i, got, want[i]);
                ok = false;
            }
        }
    }
    ar_destroy(p);
    for (int r = 0; r < N; ++r) {
        if (in[r]) (void)hipFree(in[r]);
        if (out[r]) (void)hipFree(out[r]);
    }
    std::printf("%s: %s\n", c.name, ok ? "ok" : "FAILED");
    return ok;
}

}  // namespace

int main()
{
    if (ar_version() != AR_VERSION) {
        std::printf("libar reports interface %d, this program was built against %d\n", ar_version(), AR_VERSION);
        return 1;
    }
    const Case cases[] = {
        {"ar_plan, tuner's choice, fp32, in place", false, AR_FLOAT32, AR_PROTO_AUTO, 0, 0, false},
        {"ar_plan, tuner's choice, bf16, out of place", false, AR_BFLOAT16, AR_PROTO_AUTO, 0, 0, true},
        {"ar_plan_ex, LL ring, 4 channels, fp32, out of place", true, AR_FLOAT32, AR_PROTO_LL, 4, AR_ALGO_RING, true},
        {"ar_plan_ex, LL128 ring, 3 channels, bf16, in place", true, AR_BFLOAT16, AR_PROTO_LL128, 3, AR_ALGO_RING, false},
        {"ar_plan_ex, Simple ring, 16 channels, fp32, in place", true, AR_FLOAT32, AR_PROTO_SIMPLE, 16, AR_ALGO_RING, false},
        {"ar_plan_ex, direct, fp32, out of place", true, AR_FLOAT32, AR_PROTO_AUTO, 0, AR_ALGO_DIRECT, true},
    };
    for (const Case &c : cases)
        if (!run_case(c)) return 1;
    std::printf("abi gpu check: ok\n");
    return 0;
}
