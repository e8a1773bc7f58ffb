/*
 * ar.h -- C ABI of libar, a simulated-ring AllReduce for AMD MI355X (gfx950).
 *
 * What it computes.  AllReduce-sum over N rank buffers that all live in one
 * GPU's memory: afterwards every rank's buffer holds
 *     y[i] = x_0[i] + x_1[i] + ... + x_{N-1}[i].
 * The paper steers exactly this collective: its tuner picks the algorithm
 * (ring), the protocol (LL, LL128, Simple) and the channel count for every
 * AllReduce call (paper, section 2 "NCCL and its plugin system"; section 3.3,
 * the policy programming model; section 5.3, Table 2 and Figure 2, where a
 * message-size-aware choice of ring protocol and channels beats the default).
 *
 * How.  A ring reduce-scatter followed by a ring all-gather.  Each simulated
 * rank is one group of workgroups; consecutive ranks exchange chunks through
 * FIFOs in device memory, with flags as the "link".  Segment-major layout:
 * with A = 16 / element bytes, seg = roundup(ceil(count / N), A); segment s
 * covers elements [s*seg, min((s+1)*seg, count)) and is summed along the
 * ring starting at rank s (acc = x_s, then + x_{s+1}, ... + x_{s+N-1}), each
 * addition one binary32 round-to-nearest-even operation; rank s-1 owns the
 * result and the all-gather copies it around.  The result bits therefore
 * depend only on (N, count, dtype), never on protocol, channels or chunk.
 * bf16: inputs widen exactly to fp32, partial sums travel as fp32, and the
 * owner rounds once to bf16 (round to nearest even, NaN -> 0x7FC0).
 *
 * Conventions.  All sizes are in elements unless named *_bytes.  Device
 * pointers are HIP device pointers on the current device; `stream` is a
 * hipStream_t passed as void* (NULL = the null stream).  Functions that
 * return int return AR_OK (0) or an AR_ERR_* code; functions that return a
 * pointer return NULL on error and leave the code in ar_last_error().
 * Nothing here is thread-safe for one plan: use a plan from one host thread
 * and keep at most one run of a plan in flight -- not on two streams at
 * once, not in two graph replays at once, not in a replay and an eager run
 * at once (its FIFOs and flag epochs are shared by all its runs; overlapping
 * runs corrupt each other's results or end in the watchdog).
 *
 * Ring launches on one device are ordered across streams.  A ring kernel's
 * workgroups wait on each other, so its grid needs the whole grid resident;
 * two ring grids dispatched side by side could each hold part of the device
 * while waiting for room the other occupies.  While all ring launches of a
 * device go to one stream, that stream orders them and the library adds
 * nothing.  The first ring launch on a second stream waits (on the host)
 * for all work of the device once, and from then on the library records an
 * event after every ring launch of that device (one event per device) and
 * makes a ring launch on another stream than the previous one wait for it.
 * Ring collectives of different plans therefore never overlap in time,
 * whatever streams they run on; the direct algorithm's kernels are not
 * ordered (they never wait).  Launches captured into a HIP graph are not
 * ordered this way: a graph whose replays may overlap ring launches on
 * other streams must be ordered by its caller (replay it on the stream that
 * runs the others).
 */
#ifndef AR_H
#define AR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define AR_VERSION 4
#define AR_MAX_RANKS 16
#define AR_MAX_CHANNELS 256
#define AR_MAX_WAVES 16

/* Element types. */
enum { AR_FLOAT32 = 0, AR_BFLOAT16 = 1 };

/* Protocols (paper, section 2: the tuner chooses among LL, LL128, Simple).
 *   LL     8-byte lines: 4 bytes of data + 4-byte flag in one word; the
 *          reader checks the flag in the same load that brings the data
 *          (an aligned 8-byte access is single-copy atomic).
 *   LL128  128-byte lines: 120 bytes of data + 8-byte flag.  The writer makes
 *          a line's data complete before it stores the line's flag; the
 *          reader loads whole lines and, once every flag of a batch is
 *          current, uses the data of the same load.  That relies on an
 *          assumption CDNA does not document: that one 128-byte line load
 *          never returns its data half older than its flag half.  A stale
 *          first look is re-read only after the flags alone were seen
 *          current, which is ordered; AR_PLAN_LL128_ORDERED makes every
 *          batch take that path and removes the assumption.  The built-in
 *          tuner table never picks LL128 on MI355X.
 *   Simple bulk chunks behind separate ready (tail) / free (head) counters. */
enum { AR_PROTO_AUTO = -1, AR_PROTO_LL = 0, AR_PROTO_LL128 = 1, AR_PROTO_SIMPLE = 2 };

/* Algorithms (paper section 2: the tuner chooses the algorithm, e.g. ring
 * or tree, besides protocol and channels).
 *   AR_ALGO_AUTO    no preference: a requested protocol implies the ring,
 *                   otherwise the tuner decides (no opinion = ring)
 *   AR_ALGO_RING    reduce-scatter + all-gather around the ring, through
 *                   FIFOs, under a protocol and channel count
 *   AR_ALGO_DIRECT  two-shot direct reduce: for each segment, one group of
 *                   workgroups reads that segment of every rank buffer
 *                   directly, sums it in the same chain order as the ring
 *                   (x_s + x_{s+1} + ... + x_{s+N-1}) and writes the result
 *                   to every rank; identical bits, only 2 N S bytes moved,
 *                   no flags.  Protocols do not apply; nchannels is the
 *                   number of workgroups per segment (0 = sized to the
 *                   message). */
enum { AR_ALGO_AUTO = 0, AR_ALGO_RING = 1, AR_ALGO_DIRECT = 2 };

/* Collectives (paper section 2: the tuner is consulted per collective call;
 * section 5.3 measures AllReduce and AllGather).  `count` in a plan is, for
 *   AR_COLL_ALLREDUCE      each rank's buffer: count elements in, count out;
 *   AR_COLL_REDUCESCATTER  each rank's result block: rank r sends N*count
 *                          elements and receives count, block r of the sum,
 *                          summed along the ring chain that ends at rank r
 *                          (x_{r+1} + x_{r+2} + ... + x_r, binary32 RNE);
 *   AR_COLL_ALLGATHER      each rank's contribution: rank r sends count
 *                          elements and receives N*count, [x_0 | ... | x_{N-1}].
 * ReduceScatter and AllGather need count to be a multiple of 16 bytes of
 * elements (4 fp32, 8 bf16) so every block starts on a 16-byte boundary. */
enum { AR_COLL_ALLREDUCE = 0, AR_COLL_REDUCESCATTER = 1, AR_COLL_ALLGATHER = 2 };

/* Workgroup placement: how the grid index maps to (channel c, rank r).
 *   AR_PLACE_RANK_SPREAD   block = c*N + r (consecutive ranks on different XCDs)
 *   AR_PLACE_CHANNEL_LOCAL block = r*C + c (one channel's ranks share an XCD
 *                          when C is a multiple of 8)
 * Results are identical; only speed differs. */
enum { AR_PLACE_RANK_SPREAD = 0, AR_PLACE_CHANNEL_LOCAL = 1 };

/* Status codes. */
enum {
    AR_OK = 0,
    AR_ERR_ARG = 1,          /* bad argument (NULL, range, alignment, overlap) */
    AR_ERR_UNSUPPORTED = 2,  /* valid request this library does not implement */
    AR_ERR_NOMEM = 3,        /* device or host allocation failed */
    AR_ERR_HIP = 4,          /* a HIP runtime call failed */
    AR_ERR_OCCUPANCY = 5,    /* grid cannot be co-resident on the device */
    AR_ERR_TIMEOUT = 6,      /* a flag wait exceeded the watchdog (sticky) */
    AR_ERR_STATE = 7,        /* plan is in an error state; call ar_plan_reset */
    AR_ERR_SCRATCH = 8       /* ar_run_noalloc: the request needs more memory than
                                the static scratch holds (AR_NOALLOC_SCRATCH_BYTES) */
};

/* Debug knobs (ar_plan_desc.debug_flags); zero in normal use.
 *   AR_DEBUG_SKIP_POST  channel 0 / wave 0 / rank 0 announces none of its
 *                       messages, so its successor's wait runs into the
 *                       watchdog: every wave still exits and the run reports
 *                       AR_ERR_TIMEOUT.
 *   AR_DEBUG_JITTER     pseudo-random short sleeps before flag posts, to
 *                       shake out ordering races.
 *   AR_DEBUG_CHECK_LINES  torn / stale line detector for the flag-in-line
 *                       protocols (LL, LL128; paper section 2): every writer
 *                       fills each data word of a line with a check word
 *                       derived from the message's flag and the word's byte
 *                       offset in the slot, instead of data; every reader,
 *                       once it has accepted a line by its flag (by the
 *                       normal protocol code), compares each data word of
 *                       the line with the check word that flag implies.  A
 *                       line whose data belongs to another message or
 *                       another place counts as bad.  Counts are read with
 *                       ar_plan_debug_stats.  The collective's results are
 *                       undefined in this mode.  Simple plans ignore it.
 *   AR_DEBUG_TRACE      channel 0 / wave 0 of every rank writes one record
 *                       per ring step into the buffer given by
 *                       ar_plan_debug_trace (see there).
 * A ring plan with any debug flag runs a kernel build that carries these
 * hooks; plans without them run one that does not (the hooks cost time even
 * when not taken). */
enum { AR_DEBUG_SKIP_POST = 1u, AR_DEBUG_JITTER = 2u, AR_DEBUG_CHECK_LINES = 4u, AR_DEBUG_TRACE = 8u };

typedef struct ar_plan_s ar_plan_t;

/* Full plan description.  Zero fields take the tuner's choice or the
 * library default, so a zero-initialised struct plus {nranks, count, dtype,
 * proto = AR_PROTO_AUTO} is a valid request. */
typedef struct ar_plan_desc {
    int nranks;            /* 1 .. AR_MAX_RANKS; N = 1 is a no-op */
    int dtype;             /* AR_FLOAT32 or AR_BFLOAT16 */
    size_t count;          /* elements per rank; 0 is a valid no-op */
    int proto;             /* AR_PROTO_*; AUTO asks the tuner */
    int nchannels;         /* 1 .. AR_MAX_CHANNELS; 0 asks the tuner */
    size_t chunk_bytes;    /* data bytes per ring step per (segment, channel);
                              0 asks the tuner / default */
    int fifo_depth;        /* FIFO slots per connection (2..16); 0 = default:
                              2 (Simple) or 4 (LL, LL128), doubled up to 16
                              while a run has more messages than slots and
                              the FIFO stays within 4 MiB */
    int nwaves;            /* wavefronts per workgroup (1..AR_MAX_WAVES); 0 = default */
    int placement;         /* AR_PLACE_* */
    uint32_t timeout_us;   /* watchdog per flag wait; 0 = default (2 s) */
    uint32_t debug_flags;  /* AR_DEBUG_*; 0 in normal use */
    int max_channels;      /* geometry query only: device channel capacity
                              (0 = AR_MAX_CHANNELS); plans use the device's */
    uint64_t comm_id;      /* communicator key passed to the tuner and used
                              by the profiler hook (0 if unused) */
    uint32_t flags;        /* AR_PLAN_* */
    int algo;              /* AR_ALGO_* */
    int coll;              /* AR_COLL_* (0 = AllReduce) */
    int direct_unroll;     /* direct algorithm: 1 or 2 units per thread and
                              iteration; 0 asks the tuner / default */
} ar_plan_desc;

/* Plan flags.
 *   AR_PLAN_PROFILE  record each run's kernel duration (HIP events around the
 *                    launch) into the telemetry map under desc.comm_id.  A
 *                    run's sample is harvested without blocking by a later
 *                    ar_run, or by ar_plan_status; a run whose predecessor's
 *                    events are still pending is not timed.
 *   AR_PLAN_FIFO_ONLY  ring plans: carry every hop through the FIFOs.  By
 *                    default (the peer-direct mode) the second rank of each
 *                    reduce-scatter chain reads the chain start's input
 *                    from that rank's buffer (one hop and its flag fewer),
 *                    and the Simple ring also writes each finished
 *                    all-gather chunk straight into the next rank's output
 *                    buffer and forwards it from there (nothing moves on
 *                    the last hop); the LL and LL128 all-gathers keep their
 *                    lines, whose flags cannot live in a user buffer.  The
 *                    result bits are the same either way.  The direct
 *                    algorithm has no FIFOs and ignores the flag.
 *   AR_PLAN_LL128_ORDERED  LL128 only: a reader uses a batch of lines only
 *                    from loads issued after it has seen every flag of the
 *                    batch current (it polls the 8-byte flags, then reads
 *                    the lines), never from a load that brought data and
 *                    flag together.  This takes no assumption about how a
 *                    128-byte load is served, at the cost of one more round
 *                    trip per batch.  Other protocols ignore the flag. */
enum { AR_PLAN_PROFILE = 1u, AR_PLAN_FIFO_ONLY = 2u, AR_PLAN_LL128_ORDERED = 4u };

/* Resolved plan geometry (after the tuner and defaults). */
typedef struct ar_plan_info {
    int nranks, dtype, proto, nchannels, nwaves, fifo_depth, placement;
    int grid;              /* workgroups = nchannels * nranks */
    int block;             /* threads per workgroup = 64 * nwaves */
    size_t count;
    size_t seg_elems;      /* segment length: roundup(ceil(count/N), A) */
    size_t chan_elems;     /* per-channel sub-range of a segment */
    size_t chunk_elems;    /* per-(segment, channel) ring step */
    size_t wave_elems;     /* one wave's share of a chunk step */
    size_t nchunks;        /* chunk steps per channel sub-range */
    size_t slot_bytes;     /* one FIFO slot of one (connection, wave) */
    size_t fifo_bytes;     /* all FIFO slots */
    size_t flag_bytes;     /* head/tail counters, ring epochs, control words */
    uint64_t msgs_per_run; /* messages per connection per run: nchunks*(2N-2)
                              (AllReduce) or nchunks*(N-1) (ReduceScatter /
                              AllGather); with peer_direct, nchunks fewer for
                              AllReduce and ReduceScatter */
    uint64_t wire_bytes_per_run; /* bytes that cross ring links per run (all
                              connections): written to a FIFO with flags, or,
                              with peer_direct, the chain starts' inputs read
                              by the second ranks and (Simple) all-gather
                              chunks written into the next rank's output */
    int algo;              /* AR_ALGO_RING or AR_ALGO_DIRECT */
    int coll;              /* AR_COLL_* */
    int peer_direct;       /* 1: the ring reads the chain start's input
                              directly, and the Simple ring writes all-gather
                              chunks into the next rank's output (see
                              AR_PLAN_FIFO_ONLY) */
    int direct_unroll;     /* direct algorithm: units per thread and iteration */
} ar_plan_info;

/* ---- plans -------------------------------------------------------------- */

/* Create a plan for AllReduce of `count` elements of `dtype` over `nranks`
 * simulated ranks on the current HIP device.  proto = AR_PROTO_AUTO or
 * nchannels = 0 consults the active tuner with msg_bytes = count * element
 * size.  The plan owns its FIFO, flag and status memory (device memory on
 * the current device, zeroed here, freed by ar_destroy).  Returns NULL on
 * error (see ar_last_error): AR_ERR_ARG for out-of-range arguments,
 * AR_ERR_OCCUPANCY if nchannels * nranks workgroups cannot be co-resident,
 * AR_ERR_NOMEM / AR_ERR_HIP for allocation or device failures. */
ar_plan_t *ar_plan(int nranks, size_t count, int dtype, int proto, int nchannels);

/* Same as ar_plan with every knob of ar_plan_desc. */
ar_plan_t *ar_plan_ex(const ar_plan_desc *desc);

/* In-place collective.  `bufs` is a host array of nranks device pointers,
 * 16-byte aligned and pairwise non-overlapping, each to the plan's full
 * buffer: count elements (AllReduce) or N*count elements (ReduceScatter:
 * rank r's result lands in block r of its buffer, at bufs[r] + r*count;
 * AllGather: rank r's contribution is read from block r of its buffer).
 * For AllReduce each buffer holds y on completion.  The pointer array is copied;
 * the buffers stay owned by the caller.  Enqueued asynchronously on `stream`:
 * errors found on the host are returned (AR_ERR_ARG, AR_ERR_STATE,
 * AR_ERR_HIP); a watchdog timeout inside the kernel is reported later by
 * ar_plan_status.  Safe in place: a rank reads each element of its input
 * before it writes the result to that element.  The launch carries no
 * per-run state (flag epochs live in the plan's device memory), so it may
 * be captured into a HIP graph and replayed; issues no memset. */
int ar_run(ar_plan_t *plan, void *const *bufs, void *stream);

/* Out-of-place collective: reads send[r], writes recv[r] (sizes per
 * collective as above).  recv buffers must not overlap each other or any
 * other rank's send buffer; recv[r] may equal send[r] (AllReduce) or sit at
 * send[r] + r*count (ReduceScatter) / contain send[r] at recv[r] + r*count
 * (AllGather), the in-place layouts.  Same numerics as ar_run. */
int ar_run_oop(ar_plan_t *plan, const void *const *send, void *const *recv, void *stream);

/* Bytes of the static scratch that ar_run_noalloc uses on each device. */
#define AR_NOALLOC_SCRATCH_BYTES (16u << 20)

/* Allocation-free collective, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  It runs the collective `desc` describes (as ar_plan_ex
 * would plan it: the tuner, defaults and clamps are the same) from send[r]
 * to recv[r] on `stream`, with the same numerics and buffer rules as
 * ar_run_oop, and calls no hipMalloc, hipFree, event or stream creation:
 * the ring's FIFOs, flags and control words live in a static device array
 * of AR_NOALLOC_SCRATCH_BYTES per device, which every call on that device
 * shares and which keeps the last call's contents until the process ends.
 * Each call clears the part it uses with a fill kernel on `stream` (no
 * memset), so a captured call replays correctly.  Calls whose runs overlap
 * on one device race on the array: keep them on one stream, or order them.
 * Ring launches made here are not ordered against other streams' ring
 * launches (see the conventions above); the caller orders them.
 * Errors: AR_ERR_SCRATCH when the ring's FIFO, flags and control words need
 * more than AR_NOALLOC_SCRATCH_BYTES (pick smaller chunks, fewer channels or
 * waves, or the direct algorithm, which needs no scratch); AR_ERR_UNSUPPORTED
 * for AR_PLAN_PROFILE (it needs events); otherwise as ar_plan_ex and
 * ar_run_oop.  A watchdog timeout inside the kernel makes every wave leave
 * (the output is then undefined) and is not reported: the next call clears
 * the status word.  The first call on a device looks up that device's copy
 * of the array (with the device current). */
int ar_run_noalloc(const ar_plan_desc *desc, const void *const *send, void *const *recv, void *stream);

/* Watchdog status, to be read after the stream has been synchronised:
 * AR_OK, or AR_ERR_TIMEOUT if any wave's flag wait exceeded the watchdog in
 * any run since creation or the last ar_plan_reset (sticky).  While sticky,
 * ar_run returns AR_ERR_STATE without launching. */
int ar_plan_status(ar_plan_t *plan);

/* Re-zero the plan's FIFOs, flags and status and restart its flag epoch.
 * Synchronous (waits for the device); call when no run is in flight. */
int ar_plan_reset(ar_plan_t *plan);

/* Debug: fill every FIFO data byte with 0xFF (a NaN pattern and an invalid
 * LL/LL128 flag) on `stream`, leaving the flags intact, so that a reader that
 * consumed a slot before it was written would see NaN.  Call between runs. */
int ar_plan_poison(ar_plan_t *plan, void *stream);

/* Line-check counts of AR_DEBUG_CHECK_LINES since the plan was created or
 * last reset, summed over every wave of every run. */
typedef struct ar_debug_stats {
    uint64_t lines_checked;    /* LL / LL128 lines accepted by their flag and checked */
    uint64_t lines_first_read; /* of those, accepted from the first load of the line
                                  (LL128: data and flag from one 128-byte load) */
    uint64_t lines_bad;        /* of those, with data not matching the flag */
} ar_debug_stats;

/* Read the counts (synchronous copy; call after synchronising the plan's
 * stream).  AR_ERR_ARG for NULL arguments. */
int ar_plan_debug_stats(ar_plan_t *plan, ar_debug_stats *out);

/* Give an AR_DEBUG_TRACE plan its trace buffer: `buf` is device memory of
 * `bytes` bytes owned by the caller, kept by the plan until replaced (NULL
 * stops tracing) and written by every later run.  The buffer is split into
 * equal shares per rank; rank r's k-th ring step of a run (channel 0,
 * wave 0) writes record r * per_rank + k, per_rank = bytes / (64 * nranks),
 * and steps beyond per_rank are not recorded.  A record is eight uint64_t:
 * t_begin (step entered), t_recv (first data of the step accepted: flag or
 * counter observed), polls (LL: reloads before the first batch was
 * accepted; LL128: 1 if the first look at the first batch was stale; Simple
 * 0), t_issued (the step's, for LL128 its first flag group's, data stores
 * issued), t_drained (those stores complete; LL 0), t_posted (the flag or
 * counter that publishes them stored), msg (message index sent, or taken by
 * a receive-only step), kind (the step's kind).  Times are ticks of the
 * device's 100 MHz real-time counter, common to all XCDs; fields a step
 * does not reach stay 0.  AR_ERR_ARG for a NULL plan. */
int ar_plan_debug_trace(ar_plan_t *plan, void *buf, size_t bytes);

/* Free the plan.  The caller must have synchronised every stream that ran
 * it.  NULL is ignored. */
void ar_destroy(ar_plan_t *plan);

/* Resolved geometry of an existing plan. */
int ar_plan_get_info(const ar_plan_t *plan, ar_plan_info *out);

/* Device memory the plan holds (FIFO + flags + control words), bytes. */
size_t ar_plan_workspace_bytes(const ar_plan_t *plan);

/* Resolve a description to its geometry on the host alone (tuner, defaults,
 * segment / channel / chunk split, FIFO sizes) without touching a GPU.
 * Uses desc->max_channels (0 = AR_MAX_CHANNELS) as the channel capacity. */
int ar_plan_geometry(const ar_plan_desc *desc, ar_plan_info *out);

/* ---- tuner (paper, section 3.3, policy programming model; section 4,
 *      cost-table fallback and channel clamp; section 5.3, size-aware policy) */

/* Input of a tuning decision: mirrors the paper's policy context
 * (collective type, message size, rank count) plus dtype and the channel
 * capacity the decision must respect. */
typedef struct ar_tune_ctx {
    int coll;              /* AR_COLL_* */
    size_t msg_bytes;      /* bytes of one rank's full buffer: AllReduce count *
                              element size; ReduceScatter / AllGather nranks *
                              count * element size */
    int nranks;
    int dtype;
    int max_channels;      /* the decision is clamped to [1, max_channels] */
    uint64_t comm_id;      /* caller-chosen communicator key (0 if unused) */
} ar_tune_ctx;

/* Output of a tuning decision. */
typedef struct ar_tune_out {
    int proto;             /* AR_PROTO_LL / LL128 / SIMPLE; AUTO = no opinion */
    int nchannels;         /* 0 = no opinion */
    size_t chunk_bytes;    /* 0 = protocol default */
    int nwaves;            /* 0 = protocol default */
    int algo;              /* AR_ALGO_*; AUTO = no opinion (ring).  proto,
                              nchannels, chunk_bytes and nwaves describe the
                              ring choice, used whenever the ring runs. */
    int direct_parts;      /* direct algorithm: workgroups per segment
                              (0 = sized to the message) */
    int direct_nwaves;     /* direct algorithm: waves per workgroup (0 = 4) */
    int direct_unroll;     /* direct algorithm: 16-byte units per thread and
                              iteration, 1 or 2 (0 = by size: 2 up to 8 MiB
                              per rank, 1 above) */
} ar_tune_out;

/* A tuner: fill *out from *ctx; return 0 on success.  A non-zero return, or
 * an output outside the valid ranges, makes ar_tune fall back to the fixed
 * default (Simple, 16 channels) -- the analogue of the paper's cost table,
 * where unavailable choices fall back to the library's own. */
typedef int (*ar_tuner_fn)(const ar_tune_ctx *ctx, ar_tune_out *out, void *user);

/* Make fn (with its user pointer) the active tuner; NULL restores the built-in
 * MI355X table.  The swap is one atomic pointer exchange (paper section 4,
 * hot reload): a decision already in progress finishes with the old tuner,
 * the next one uses the new tuner, and no decision is lost.  Returns after
 * every decision that was using the old tuner has finished, so the caller may
 * then release the old tuner's code and data.  Thread-safe against
 * concurrent ar_tune calls; concurrent swaps are serialised by the exchange
 * (each one drains the tuner it replaced).  Must not be called from inside a
 * tuner (it would wait for its own decision).  AR_ERR_NOMEM if the slot for
 * the new tuner cannot be allocated. */
int ar_set_tuner(ar_tuner_fn fn, void *user);

/* Timings of one reload, nanoseconds. */
typedef struct ar_reload_stats {
    uint64_t validate_ns;  /* probing the candidate on the context grid */
    uint64_t swap_ns;      /* the atomic exchange itself */
    uint64_t drain_ns;     /* waiting for decisions still using the old tuner */
    uint64_t probes;       /* contexts the candidate was called on */
} ar_reload_stats;

/* Checked hot reload (paper section 3.1 T1/T3, section 4): first call the
 * candidate on a fixed grid of contexts (message sizes 0 B .. 1 GiB, 1..16
 * ranks, both dtypes, several channel capacities); if any call returns
 * non-zero or a malformed decision (unknown protocol, negative channels or
 * waves, waves > AR_MAX_WAVES, chunk > 64 MiB), return AR_ERR_ARG and keep
 * the current tuner untouched.  Otherwise behave as ar_set_tuner.  stats may
 * be NULL.  A well-formed tuner that makes poor choices is accepted. */
int ar_reload_tuner(ar_tuner_fn fn, void *user, ar_reload_stats *stats);

/* Run the active tuner on *ctx, validate and clamp, and write a complete
 * decision to *out (proto, nchannels, chunk_bytes and nwaves all set).
 * Returns AR_ERR_ARG for a NULL or invalid ctx; otherwise AR_OK, also when
 * the tuner's answer was replaced by the fallback. */
int ar_tune(const ar_tune_ctx *ctx, ar_tune_out *out);

/* Built-in tuners. */
/* ar_tuner_table: measured MI355X tables, one row per power-of-two size
 * bucket of msg_bytes (4 KiB .. 128 MiB), one table per collective and data
 * type (bf16 reduce-scatter hops carry fp32 partials, which moves the best
 * geometry).  Every row was measured with 8 ranks.  For N ranks a row's
 * channel and direct part counts are scaled by 8 / N (rounded, at least
 * 1), so that the grid keeps the workgroup count the row was measured
 * with; with two ranks the LL rows defer to the default, whose peer-direct
 * Simple ring waits for no flag at all there.  Results are identical for
 * every choice.  Collectives outside the tables defer to the default. */
int ar_tuner_table(const ar_tune_ctx *ctx, ar_tune_out *out, void *user);
int ar_tuner_fixed_default(const ar_tune_ctx *ctx, ar_tune_out *out, void *user); /* Simple, 16 channels */
int ar_tuner_noop(const ar_tune_ctx *ctx, ar_tune_out *out, void *user);          /* defers: no opinion */

/* ---- telemetry and the adaptive tuner (paper section 3.3, Listing 1: a
 *      profiler writes latency into a shared typed map that the tuner reads;
 *      section 5.3, composability) ----------------------------------------- */

/* Latest sample of one communicator. */
typedef struct ar_latency_state {
    uint64_t comm_id;
    uint64_t latency_ns;   /* duration of the sampled run (saturates at 2^48-1) */
    int nchannels;         /* channel count the sampled run used */
    uint64_t samples;      /* samples recorded for this communicator */
} ar_latency_state;

/* Profiler hook: store (latency_ns, nchannels) as the latest sample of
 * comm_id in the fixed-size telemetry map (1024 communicators).  Thread-safe.
 * AR_ERR_ARG for nchannels outside 0..65535, AR_ERR_NOMEM if the map is
 * full. */
int ar_profile_record(uint64_t comm_id, uint64_t latency_ns, int nchannels);

/* Look up comm_id's latest sample; AR_ERR_ARG if it has none (callers must
 * check, as a map lookup can come back empty). */
int ar_profile_lookup(uint64_t comm_id, ar_latency_state *out);

/* Forget every communicator (tuner state included).  Call only while no
 * other thread records, looks up or tunes. */
void ar_profile_clear(void);

/* Configuration of ar_tuner_adaptive (its user pointer; NULL = defaults
 * {2, 12, 9000, 4, AR_PROTO_SIMPLE}: 2 -> 12 channels in 90,000 decisions). */
typedef struct ar_adaptive_cfg {
    int min_channels;      /* conservative start and back-off level */
    int max_channels;      /* ramp ceiling */
    uint32_t ramp_calls;   /* uncontended decisions per +1 channel */
    uint32_t backoff_ratio;/* contended when latency > ratio x the fastest
                              latency seen at the same or fewer channels */
    int proto;             /* protocol of every decision */
} ar_adaptive_cfg;

/* Closed-loop channel tuner over the telemetry of ctx->comm_id: with no
 * samples it answers min_channels; otherwise it backs off to min_channels
 * when the latest sample is contended and adds one channel every ramp_calls
 * uncontended decisions up to max_channels.  Returns -1 (so ar_tune falls
 * back) for an invalid configuration. */
int ar_tuner_adaptive(const ar_tune_ctx *ctx, ar_tune_out *out, void *user);

/* The paper's Listing 1 closed-loop policy (section 3.3) over the same
 * telemetry: no sample for ctx->comm_id -> 4 channels and no other opinion
 * (ar_tune then applies the default: the Simple ring); with a sample,
 * messages of at most 32 KiB take the small-message algorithm (here
 * AR_ALGO_DIRECT, in place of the listing's tree), larger ones the ring,
 * with the Simple protocol, and when the last sample's latency exceeds
 * 1 ms, one channel more than that run used (at most 16), otherwise the
 * same count.  user is unused. */
int ar_tuner_size_adaptive(const ar_tune_ctx *ctx, ar_tune_out *out, void *user);

/* ---- errors and version ------------------------------------------------- */

const char *ar_strerror(int code);
int ar_last_error(void);   /* code of the last failed call on this thread */
int ar_version(void);

/* ---- device self-checks ------------------------------------------------- */

/* Round n floats to bf16 bits with the library's device conversion (round to
 * nearest even, NaN -> 0x7FC0): in and out are device pointers, enqueued on
 * stream.  Lets tests compare the device rounding with other conversions. */
int ar_debug_bf16_round(const float *in, uint16_t *out, size_t n, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* AR_H */
