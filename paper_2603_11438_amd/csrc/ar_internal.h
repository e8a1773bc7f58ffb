// Internal declarations shared by the host runtime and the HIP kernels of
// libar.  Not part of the C ABI (see include/ar.h).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "ar.h"

namespace ar {

// Flag memory layout: every connection (channel c, wave w, sender rank r,
// i.e. the link r -> r+1 of one wave's ring) owns two 128-byte lines, so no
// two counters written by different waves share a cache line.
//   tail: messages the sender has published on the link (sender writes)
//   head: messages the receiver has consumed on the link (receiver writes)
// The sender's tail line also holds, at u64 offset kEpochU64, that wave's
// message epoch: the absolute index of its next run's first message.
constexpr int kFlagLineU64 = 16;                 // 128 bytes
constexpr int kConnFlagU64 = 2 * kFlagLineU64;   // tail line + head line
constexpr int kEpochU64 = 8;                     // epoch: byte 64 of the tail line
constexpr int kCtlU32 = 64;                      // control block: 256 bytes
constexpr int kCtlAbort = 0;                     // nonzero: every wave must leave
constexpr int kCtlStatus = 32;                   // sticky AR_ERR_* bit set
// Line-check counters of AR_DEBUG_CHECK_LINES, 64-bit, at these u32 indices
// (bytes 64..87, a line of their own).
constexpr int kCtlLinesChecked = 16;             // LL / LL128 lines accepted and checked
constexpr int kCtlLinesFirst = 18;               // of those, accepted on the first load
constexpr int kCtlLinesBad = 20;                 // of those, data not matching the flag
// A step record of AR_DEBUG_TRACE: this many 64-bit fields.
constexpr int kTraceFields = 8;

// Status bits written by the kernel into ctl[kCtlStatus].
constexpr uint32_t kStatusTimeout = 1u;

// Everything a ring kernel launch needs; passed by value as the kernel
// argument.  Counts are in elements of the plan's dtype.
struct RingArgs {
    const char *src[AR_MAX_RANKS];   // rank inputs
    char *dst[AR_MAX_RANKS];         // rank outputs (== src for in place)
    char *fifo;                      // all FIFO slots
    uint64_t *flags;                 // per-connection head/tail lines
    uint32_t *ctl;                   // abort word + status word
    uint64_t count;                  // elements of the segmented buffer (AllReduce: count;
                                     // ReduceScatter / AllGather: N blocks of count)
    uint64_t seg;                    // segment length (ReduceScatter / AllGather: one block)
    uint64_t cs;                     // per-channel sub-range of a segment
    uint64_t chunk;                  // per-(segment, channel) ring step
    uint64_t kw;                     // one wave's share of a chunk step
    uint64_t part;                   // elements of segment full_segs (0 .. seg-1)
    uint64_t slot_bytes;             // bytes of one FIFO slot
    uint64_t timeout_ticks;          // watchdog, in 100 MHz real-time ticks
    uint32_t nranks, nchannels, nwaves, depth, nchunks, placement, debug;
    uint32_t ll128_ordered;          // AR_PLAN_LL128_ORDERED: lines only from loads after their flags
    uint32_t coll;                   // AR_COLL_*: which steps of the ring run
    uint32_t full_segs;              // segments 0 .. full_segs-1 hold seg elements; segment
                                     // full_segs holds part, any later one none
    uint64_t *trace;                 // AR_DEBUG_TRACE: step records, rank r's at
                                     // [r * trace_per_rank, (r + 1) * trace_per_rank)
    uint32_t trace_per_rank;         // records per rank (0: none kept)
};

// Resolved plan geometry.  Computed on the host only.
int resolve_geometry(const ar_plan_desc *desc, int max_channels, ar_plan_info *out);

// Protocol defaults.
int default_nwaves(int proto);
int default_depth(int proto);
size_t default_chunk_bytes(int proto);

// Kernel launchers (ar_kernels.hip).
int launch_ring(const ar_plan_info &info, const RingArgs &args, void *stream);
int launch_fill_u32(uint32_t *p, size_t n, uint32_t value, void *stream);
int launch_copy(const void *src, void *dst, size_t bytes, void *stream);
int ring_occupancy(int proto, int dtype, int block, int *blocks_per_cu);
int launch_bf16_round(const float *in, uint16_t *out, size_t n, void *stream);

// Run-time helpers of ar_runtime.cpp.
constexpr uint32_t kDefaultTimeoutUs = 2000000;  // 2 s per flag wait
constexpr uint64_t kTicksPerUs = 100;            // 100 MHz real-time counter
// Bytes of each rank's send and recv buffer for a collective's geometry.
void buffer_bytes(const ar_plan_info &g, size_t *send_b, size_t *recv_b);
// Rank buffers non-NULL, 16-byte aligned, receive buffers overlapping
// nothing but their own rank's in-place layout: AR_OK or AR_ERR_ARG.
int check_buffers(const ar_plan_info &g, const void *const *send, void *const *recv);
// Workgroups of a ring launch that fit on the current device, per rank.
int device_channel_capacity(int proto, int dtype, int nranks, int nwaves, int *cap);
// Kernel arguments of one run.
void fill_args(const ar_plan_info &g, const ar_plan_desc &d, uint64_t timeout_ticks, const void *const *send,
               void *const *recv, char *fifo, uint64_t *flags, uint32_t *ctl, RingArgs *out);
// The tuner's and defaults' geometry for a description on the current device.
int resolve_for_device(const ar_plan_desc *desc, ar_plan_desc *d_out, ar_plan_info *info_out, int *dev_out);
// Ring memory layout: total bytes, with the flag lines and FIFO offsets.
size_t workspace_layout(const ar_plan_info &info, size_t *flags_off, size_t *fifo_off);

// Thread-local last error.
void set_last_error(int code);

}  // namespace ar
