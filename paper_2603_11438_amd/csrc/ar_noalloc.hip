// Allocation-free entry point of libar (ar_run_noalloc, C ABI in ar.h): the
// ring's FIFOs, flags and control words live in a static device array
// instead of a plan's hipMalloc'd workspace.
#include <hip/hip_runtime.h>

#include <mutex>
#include <stdint.h>
#include <string.h>

#include "ar.h"
#include "ar_internal.h"

using namespace ar;

// The static scratch.  Each device that loads the library holds its own copy
// until the process ends.  In host code this name stands for a host-side
// shadow, not a device address: passing it to a kernel would make the
// kernel fault.  The address each device gives it is fetched once per device
// (scratch_of) and only that address reaches kernels and fills.
static __device__ __align__(256) unsigned char scratch[AR_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kScratchBytes = AR_NOALLOC_SCRATCH_BYTES;
constexpr int kScratchMaxDevices = 64;

std::mutex g_scratch_mu;
void *g_scratch_ptr[kScratchMaxDevices];

// Device address of `device`'s copy of the scratch; looked up on the first
// call for that device, which is the current device (the caller checked).
int scratch_of(int device, void **ptr)
{
    if (device < 0 || device >= kScratchMaxDevices) return AR_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return AR_ERR_HIP;
        if (((uintptr_t)p & 255u) != 0) return AR_ERR_HIP;
        g_scratch_ptr[device] = p;
    }
    *ptr = g_scratch_ptr[device];
    return AR_OK;
}

int ret(int code)
{
    if (code != AR_OK) set_last_error(code);
    return code;
}

}  // namespace

extern "C" int ar_run_noalloc(const ar_plan_desc *desc, const void *const *send, void *const *recv, void *stream)
{
    if (!desc) return ret(AR_ERR_ARG);
    // Per-run timing needs events, which a caller that cannot allocate
    // cannot have created.
    if (desc->flags & AR_PLAN_PROFILE) return ret(AR_ERR_UNSUPPORTED);
    ar_plan_desc d;
    ar_plan_info g;
    int dev = 0;
    int rc = resolve_for_device(desc, &d, &g, &dev);
    if (rc != AR_OK) return ret(rc);
    rc = check_buffers(g, send, recv);
    if (rc != AR_OK) return ret(rc);
    const size_t bytes = g.count * (g.dtype == AR_FLOAT32 ? 4 : 2);
    if (bytes == 0) return AR_OK;
    if (g.grid == 0) return ret(launch_copy(send[0], recv[0], bytes, stream));
    const uint32_t tus = d.timeout_us ? d.timeout_us : kDefaultTimeoutUs;
    RingArgs a;
    if (g.algo != AR_ALGO_RING) {
        // The direct algorithm uses no memory besides the rank buffers.
        fill_args(g, d, (uint64_t)tus * kTicksPerUs, send, recv, nullptr, nullptr, nullptr, &a);
        return ret(launch_ring(g, a, stream));
    }
    size_t flags_off = 0, fifo_off = 0;
    const size_t need = workspace_layout(g, &flags_off, &fifo_off);
    if (need > kScratchBytes) return ret(AR_ERR_SCRATCH);
    void *base = nullptr;
    rc = scratch_of(dev, &base);
    if (rc != AR_OK) return ret(rc);
    char *ws = (char *)base;
    // The array keeps the last call's contents.  Every run starts from zeroed
    // control words, counters, epochs and FIFO lines (a stale LL or LL128
    // line of the last call could carry this call's first flags), cleared
    // by a fill kernel in stream order so that a graph capture records it
    // as a kernel node.
    rc = launch_fill_u32((uint32_t *)ws, need / 4, 0u, stream);
    if (rc != AR_OK) return ret(rc);
    fill_args(g, d, (uint64_t)tus * kTicksPerUs, send, recv, ws + fifo_off,
              (uint64_t *)(ws + flags_off), (uint32_t *)ws, &a);
    return ret(launch_ring(g, a, stream));
}

