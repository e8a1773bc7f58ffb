// Plan lifetime, argument checking and launches of libar (C ABI in ar.h).
#include <hip/hip_runtime.h>

#include <new>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "ar.h"
#include "ar_internal.h"
#include "ring_gate.h"

using namespace ar;

struct ar_plan_s {
    ar_plan_info info;
    ar_plan_desc desc;
    int device;
    char *ws;            // one allocation: control block, flags, FIFO
    size_t ws_bytes;
    uint32_t *ctl;
    uint64_t *flags;
    char *fifo;
    uint64_t timeout_ticks;
    int sticky;          // host-side copy of a timeout seen by ar_plan_status
    // Profiler hook (AR_PLAN_PROFILE): one pair of events around the last
    // timed launch, harvested without blocking.
    hipEvent_t ev_start, ev_stop;
    bool ev_pending;
    // AR_DEBUG_TRACE: the caller's record buffer.
    uint64_t *trace;
    uint32_t trace_per_rank;
};

namespace {

template <typename T>
T *fail(int code)
{
    set_last_error(code);
    return nullptr;
}

int ret(int code)
{
    if (code != AR_OK) set_last_error(code);
    return code;
}

size_t round_up(size_t a, size_t b) { return (a + b - 1) / b * b; }

bool overlap2(uintptr_t a, size_t na, uintptr_t b, size_t nb) { return a < b + nb && b < a + na; }

}  // namespace

namespace ar {

// Bytes of each rank's send and recv buffer for the plan's collective.
void buffer_bytes(const ar_plan_info &g, size_t *send_b, size_t *recv_b)
{
    const size_t blk = g.count * (g.dtype == AR_FLOAT32 ? 4 : 2);
    const size_t full = g.coll == AR_COLL_ALLREDUCE ? blk : blk * (size_t)g.nranks;
    *send_b = g.coll == AR_COLL_ALLGATHER ? blk : full;
    *recv_b = g.coll == AR_COLL_REDUCESCATTER ? blk : full;
}

// Validate rank buffers: non-NULL, 16-byte aligned, and no recv buffer
// overlapping another rank's send or recv buffer.  A rank's own send and
// recv buffers may coincide only in the collective's in-place layout.
int check_buffers(const ar_plan_info &g, const void *const *send, void *const *recv)
{
    if (!send || !recv) return AR_ERR_ARG;
    const int n = g.nranks;
    size_t sb, rb;
    buffer_bytes(g, &sb, &rb);
    if (sb == 0) return AR_OK;
    const size_t blk = g.count * (g.dtype == AR_FLOAT32 ? 4 : 2);
    for (int r = 0; r < n; ++r) {
        if (!send[r] || !recv[r]) return AR_ERR_ARG;
        if (((uintptr_t)send[r] | (uintptr_t)recv[r]) & 15u) return AR_ERR_ARG;
        const uintptr_t s = (uintptr_t)send[r], d = (uintptr_t)recv[r];
        bool in_place = false;
        if (g.coll == AR_COLL_ALLREDUCE) in_place = s == d;
        else if (g.coll == AR_COLL_REDUCESCATTER) in_place = d == s + (size_t)r * blk;
        else in_place = s == d + (size_t)r * blk;
        if (!in_place && overlap2(s, sb, d, rb)) return AR_ERR_ARG;
    }
    for (int r = 0; r < n; ++r) {
        for (int q = 0; q < n; ++q) {
            if (q == r) continue;
            if (overlap2((uintptr_t)recv[r], rb, (uintptr_t)recv[q], rb)) return AR_ERR_ARG;
            if (overlap2((uintptr_t)recv[r], rb, (uintptr_t)send[q], sb)) return AR_ERR_ARG;
        }
    }
    return AR_OK;
}

int device_channel_capacity(int proto, int dtype, int nranks, int nwaves, int *cap)
{
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return AR_ERR_HIP;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return AR_ERR_HIP;
    int rc = ring_occupancy(proto, dtype, 64 * nwaves, &per_cu);
    if (rc != AR_OK) return rc;
    long total = (long)per_cu * cus;
    long ch = total / nranks;
    if (ch > AR_MAX_CHANNELS) ch = AR_MAX_CHANNELS;
    *cap = (int)ch;
    return AR_OK;
}

}  // namespace ar

namespace {

// HIP side of the ring launch gate (ring_gate.h).
struct HipGateApi {
    using Stream = hipStream_t;
    using Event = hipEvent_t;
    static int capturing(Stream s, bool *yes)
    {
        hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(s, &st) != hipSuccess) return AR_ERR_HIP;
        *yes = st != hipStreamCaptureStatusNone;
        return 0;
    }
    static int sync_device() { return hipDeviceSynchronize() == hipSuccess ? 0 : AR_ERR_HIP; }
    // Ordering kernels of one device needs no system-scope release.
    static int create(Event *e)
    {
        return hipEventCreateWithFlags(e, hipEventDisableTiming | hipEventDisableSystemFence) == hipSuccess
                   ? 0 : AR_ERR_HIP;
    }
    static int wait(Stream s, Event e) { return hipStreamWaitEvent(s, e, 0) == hipSuccess ? 0 : AR_ERR_HIP; }
    static int record(Event e, Stream s) { return hipEventRecord(e, s) == hipSuccess ? 0 : AR_ERR_HIP; }
};

RingGate<HipGateApi> g_ring_gate;

}  // namespace

namespace ar {

// Everything a launch needs besides the plan's memory.
void fill_args(const ar_plan_info &g, const ar_plan_desc &d, uint64_t timeout_ticks, const void *const *send,
               void *const *recv, char *fifo, uint64_t *flags, uint32_t *ctl, RingArgs *out)
{
    RingArgs a;
    memset(&a, 0, sizeof a);
    for (int r = 0; r < g.nranks; ++r) {
        a.src[r] = (const char *)send[r];
        a.dst[r] = (char *)recv[r];
    }
    a.fifo = fifo;
    a.flags = flags;
    a.ctl = ctl;
    a.count = g.coll == AR_COLL_ALLREDUCE ? g.count : g.count * (uint64_t)g.nranks;
    a.seg = g.seg_elems;
    {
        uint64_t full = a.seg ? a.count / a.seg : 0;
        if (full > (uint64_t)g.nranks) full = (uint64_t)g.nranks;
        a.full_segs = (uint32_t)full;
        a.part = full < (uint64_t)g.nranks ? a.count - full * a.seg : 0;
    }
    a.coll = (uint32_t)g.coll;
    a.cs = g.chan_elems;
    a.chunk = g.chunk_elems;
    a.kw = g.wave_elems;
    a.slot_bytes = g.slot_bytes;
    a.timeout_ticks = timeout_ticks;
    a.nranks = (uint32_t)g.nranks;
    a.nchannels = (uint32_t)g.nchannels;
    a.nwaves = (uint32_t)g.nwaves;
    a.depth = (uint32_t)g.fifo_depth;
    a.nchunks = (uint32_t)g.nchunks;
    a.placement = (uint32_t)g.placement;
    a.debug = d.debug_flags;
    a.ll128_ordered = (d.flags & AR_PLAN_LL128_ORDERED) ? 1u : 0u;
    *out = a;
}

}  // namespace ar

namespace {

// Launch a ring or direct kernel.  A ring launch goes through the device's
// gate, which keeps ring grids of different streams from overlapping.
int launch_gated(int dev, const ar_plan_info &g, const RingArgs &a, void *stream)
{
    if (g.algo != AR_ALGO_RING) return launch_ring(g, a, stream);
    RingGate<HipGateApi>::Ticket t;
    int rc = g_ring_gate.before(dev, (hipStream_t)stream, t);
    if (rc != 0) return AR_ERR_HIP;
    rc = launch_ring(g, a, stream);
    if (rc != AR_OK) return rc;
    return g_ring_gate.after(t) == 0 ? AR_OK : AR_ERR_HIP;
}

}  // namespace

namespace ar {

// Resolve a description for the current device: the tuner's choice under
// the device's channel capacity, re-checked for the resolved protocol and
// wave count.  *d receives the description the geometry was resolved from.
int resolve_for_device(const ar_plan_desc *desc, ar_plan_desc *d_out, ar_plan_info *info_out, int *dev_out)
{
    ar_plan_desc d = *desc;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return AR_ERR_HIP;

    // Channel capacity for the tuner: co-resident workgroups / nranks, for
    // the wave count the request implies (the default when the tuner picks).
    int cap = AR_MAX_CHANNELS;
    if (d.nranks >= 1 && d.nranks <= AR_MAX_RANKS && (d.dtype == AR_FLOAT32 || d.dtype == AR_BFLOAT16)) {
        int probe_proto = d.proto == AR_PROTO_AUTO ? AR_PROTO_SIMPLE : d.proto;
        if (probe_proto != AR_PROTO_LL && probe_proto != AR_PROTO_LL128 && probe_proto != AR_PROTO_SIMPLE)
            return AR_ERR_ARG;
        int rc = device_channel_capacity(probe_proto, d.dtype, d.nranks,
                                         d.nwaves > 0 && d.nwaves <= AR_MAX_WAVES ? d.nwaves : default_nwaves(probe_proto),
                                         &cap);
        if (rc != AR_OK) return rc;
        if (cap < 1) return AR_ERR_OCCUPANCY;
    }
    ar_plan_info info;
    int rc = resolve_geometry(&d, cap, &info);
    if (rc != AR_OK) return rc;
    if (info.grid > 0 && info.algo == AR_ALGO_RING) {
        // Re-check co-residency for the resolved protocol and wave count.
        int cap2 = 0;
        rc = device_channel_capacity(info.proto, info.dtype, info.nranks, info.nwaves, &cap2);
        if (rc != AR_OK) return rc;
        if (info.nchannels > cap2) {
            if (d.nchannels != 0) return AR_ERR_OCCUPANCY;
            d.nchannels = cap2;
            d.proto = info.proto;
            d.chunk_bytes = info.chunk_elems * (info.dtype == AR_FLOAT32 ? 4 : 2);
            d.nwaves = info.nwaves;
            rc = resolve_geometry(&d, cap2, &info);
            if (rc != AR_OK) return rc;
        }
    }
    *d_out = d;
    *info_out = info;
    *dev_out = dev;
    return AR_OK;
}

// Bytes of the ring's device memory: control block, flag lines, FIFO, each
// part starting on a 256-byte boundary.
size_t workspace_layout(const ar_plan_info &info, size_t *flags_off, size_t *fifo_off)
{
    const size_t ctl_bytes = kCtlU32 * 4;
    const size_t flag_bytes = round_up(info.flag_bytes - kCtlU32 * 4, 256);
    *flags_off = ctl_bytes;
    *fifo_off = ctl_bytes + flag_bytes;
    return ctl_bytes + flag_bytes + info.fifo_bytes;
}

}  // namespace ar

namespace {

// Zero device memory and wait for it, without waiting for the rest of the
// device: the fill goes to a stream of its own, which the host waits for.
int zero_and_wait(void *p, size_t bytes)
{
    hipStream_t s = nullptr;
    if (hipStreamCreateWithFlags(&s, hipStreamNonBlocking) != hipSuccess) return AR_ERR_HIP;
    int rc = AR_OK;
    if (hipMemsetAsync(p, 0, bytes, s) != hipSuccess || hipStreamSynchronize(s) != hipSuccess) rc = AR_ERR_HIP;
    if (hipStreamDestroy(s) != hipSuccess) rc = AR_ERR_HIP;
    return rc;
}

// If the last timed run has finished, record its duration as the plan's
// latest telemetry sample.  Never blocks.
void harvest_profile(ar_plan_t *p)
{
    if (!p->ev_pending) return;
    if (hipEventQuery(p->ev_stop) != hipSuccess) return;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p->ev_start, p->ev_stop) == hipSuccess && ms >= 0.f)
        (void)ar_profile_record(p->desc.comm_id, (uint64_t)((double)ms * 1e6), p->info.nchannels);
    p->ev_pending = false;
}

int run_impl(ar_plan_t *p, const void *const *send, void *const *recv, void *stream)
{
    if (!p) return ret(AR_ERR_ARG);
    if (p->sticky) return ret(AR_ERR_STATE);
    int rc = check_buffers(p->info, send, recv);
    if (rc != AR_OK) return ret(rc);
    const ar_plan_info &g = p->info;
    const size_t bytes = g.count * (g.dtype == AR_FLOAT32 ? 4 : 2);
    if (bytes == 0) return AR_OK;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev != p->device) return ret(AR_ERR_ARG);
    if (g.grid == 0) {
        // One rank: every collective is a copy of its one block.
        rc = launch_copy(send[0], recv[0], bytes, stream);
        return ret(rc);
    }
    RingArgs a;
    fill_args(g, p->desc, p->timeout_ticks, send, recv, p->fifo, p->flags, p->ctl, &a);
    a.trace = p->trace;
    a.trace_per_rank = p->trace ? p->trace_per_rank : 0;
    bool timed = false;
    if (p->desc.flags & AR_PLAN_PROFILE) {
        harvest_profile(p);
        if (!p->ev_pending && hipEventRecord(p->ev_start, (hipStream_t)stream) == hipSuccess) timed = true;
    }
    rc = launch_gated(dev, g, a, stream);
    if (rc != AR_OK) return ret(rc);
    if (timed && hipEventRecord(p->ev_stop, (hipStream_t)stream) == hipSuccess) p->ev_pending = true;
    return AR_OK;
}

}  // namespace

extern "C" {

ar_plan_t *ar_plan_ex(const ar_plan_desc *desc)
{
    if (!desc) return fail<ar_plan_t>(AR_ERR_ARG);
    ar_plan_desc d;
    ar_plan_info info;
    int dev = 0;
    int rc = resolve_for_device(desc, &d, &info, &dev);
    if (rc != AR_OK) return fail<ar_plan_t>(rc);

    ar_plan_t *p = new (std::nothrow) ar_plan_t;
    if (!p) return fail<ar_plan_t>(AR_ERR_NOMEM);
    memset(p, 0, sizeof *p);
    p->info = info;
    p->desc = d;
    p->device = dev;
    const uint32_t tus = d.timeout_us ? d.timeout_us : kDefaultTimeoutUs;
    p->timeout_ticks = (uint64_t)tus * kTicksPerUs;
    if (d.flags & AR_PLAN_PROFILE) {
        if (hipEventCreate(&p->ev_start) != hipSuccess || hipEventCreate(&p->ev_stop) != hipSuccess) {
            delete p;
            return fail<ar_plan_t>(AR_ERR_HIP);
        }
    }
    if (info.grid > 0 && info.algo == AR_ALGO_RING) {
        size_t flags_off = 0, fifo_off = 0;
        p->ws_bytes = workspace_layout(info, &flags_off, &fifo_off);
        if (hipMalloc((void **)&p->ws, p->ws_bytes) != hipSuccess) {
            delete p;
            return fail<ar_plan_t>(AR_ERR_NOMEM);
        }
        p->ctl = (uint32_t *)p->ws;
        p->flags = (uint64_t *)(p->ws + flags_off);
        p->fifo = p->ws + fifo_off;
        // The workspace must read as zeros before the first run on any
        // stream; the zeroing waits for itself, not for the whole device.
        if (zero_and_wait(p->ws, p->ws_bytes) != AR_OK) {
            (void)hipFree(p->ws);
            delete p;
            return fail<ar_plan_t>(AR_ERR_HIP);
        }
    }
    return p;
}

ar_plan_t *ar_plan(int nranks, size_t count, int dtype, int proto, int nchannels)
{
    ar_plan_desc d;
    memset(&d, 0, sizeof d);
    d.nranks = nranks;
    d.count = count;
    d.dtype = dtype;
    d.proto = proto;
    d.nchannels = nchannels;
    return ar_plan_ex(&d);
}

int ar_run(ar_plan_t *plan, void *const *bufs, void *stream)
{
    if (!plan || !bufs) return ret(AR_ERR_ARG);
    if (plan->info.coll == AR_COLL_ALLREDUCE) return run_impl(plan, (const void *const *)bufs, bufs, stream);
    // ReduceScatter / AllGather in place: the block of rank r sits at r*count.
    const int n = plan->info.nranks;
    const size_t blk = plan->info.count * (plan->info.dtype == AR_FLOAT32 ? 4 : 2);
    // Empty blocks: a no-op whatever the pointers (as for AllReduce).
    if (blk == 0) return run_impl(plan, (const void *const *)bufs, bufs, stream);
    const void *send[AR_MAX_RANKS];
    void *recv[AR_MAX_RANKS];
    for (int r = 0; r < n; ++r) {
        if (!bufs[r]) return ret(AR_ERR_ARG);
        char *b = (char *)bufs[r];
        if (plan->info.coll == AR_COLL_REDUCESCATTER) {
            send[r] = b;
            recv[r] = b + (size_t)r * blk;
        } else {
            send[r] = b + (size_t)r * blk;
            recv[r] = b;
        }
    }
    return run_impl(plan, send, recv, stream);
}

int ar_run_oop(ar_plan_t *plan, const void *const *send, void *const *recv, void *stream)
{
    return run_impl(plan, send, recv, stream);
}

int ar_plan_status(ar_plan_t *p)
{
    if (!p) return ret(AR_ERR_ARG);
    harvest_profile(p);
    if (p->sticky) return AR_ERR_TIMEOUT;
    if (!p->ctl) return AR_OK;
    uint32_t st = 0;
    if (hipMemcpy(&st, p->ctl + kCtlStatus, sizeof st, hipMemcpyDeviceToHost) != hipSuccess) return ret(AR_ERR_HIP);
    if (st & kStatusTimeout) {
        p->sticky = 1;
        return AR_ERR_TIMEOUT;
    }
    return AR_OK;
}

int ar_plan_reset(ar_plan_t *p)
{
    if (!p) return ret(AR_ERR_ARG);
    if (p->ws) {
        if (hipDeviceSynchronize() != hipSuccess) return ret(AR_ERR_HIP);
        if (hipMemset(p->ws, 0, p->ws_bytes) != hipSuccess) return ret(AR_ERR_HIP);
        if (hipDeviceSynchronize() != hipSuccess) return ret(AR_ERR_HIP);
    }
    p->sticky = 0;
    return AR_OK;
}

int ar_plan_poison(ar_plan_t *p, void *stream)
{
    if (!p) return ret(AR_ERR_ARG);
    if (!p->fifo || p->info.fifo_bytes == 0) return AR_OK;
    return ret(launch_fill_u32((uint32_t *)p->fifo, p->info.fifo_bytes / 4, 0xFFFFFFFFu, stream));
}

int ar_plan_debug_stats(ar_plan_t *p, ar_debug_stats *out)
{
    if (!p || !out) return ret(AR_ERR_ARG);
    memset(out, 0, sizeof *out);
    if (!p->ctl) return AR_OK;
    uint64_t v[3] = {0, 0, 0};
    if (hipMemcpy(v, p->ctl + kCtlLinesChecked, sizeof v, hipMemcpyDeviceToHost) != hipSuccess) return ret(AR_ERR_HIP);
    out->lines_checked = v[0];
    out->lines_first_read = v[1];
    out->lines_bad = v[2];
    return AR_OK;
}

int ar_plan_debug_trace(ar_plan_t *p, void *buf, size_t bytes)
{
    if (!p) return ret(AR_ERR_ARG);
    const size_t per = buf ? bytes / ((size_t)kTraceFields * 8 * (size_t)p->info.nranks) : 0;
    if (buf && ((uintptr_t)buf & 7u)) return ret(AR_ERR_ARG);
    p->trace = per ? (uint64_t *)buf : nullptr;
    p->trace_per_rank = per > 0xFFFFFFFFu ? 0xFFFFFFFFu : (uint32_t)per;
    return AR_OK;
}

void ar_destroy(ar_plan_t *p)
{
    if (!p) return;
    if (p->ev_start) (void)hipEventDestroy(p->ev_start);
    if (p->ev_stop) (void)hipEventDestroy(p->ev_stop);
    if (p->ws) (void)hipFree(p->ws);
    delete p;
}

int ar_plan_get_info(const ar_plan_t *p, ar_plan_info *out)
{
    if (!p || !out) return ret(AR_ERR_ARG);
    *out = p->info;
    return AR_OK;
}

size_t ar_plan_workspace_bytes(const ar_plan_t *p) { return p ? p->ws_bytes : 0; }

int ar_debug_bf16_round(const float *in, uint16_t *out, size_t n, void *stream)
{
    if (n && (!in || !out)) return ret(AR_ERR_ARG);
    return ret(launch_bf16_round(in, out, n, stream));
}

}  // extern "C"
