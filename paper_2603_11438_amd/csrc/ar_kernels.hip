// Ring AllReduce kernels for gfx950 (MI355X): reduce-scatter then
// all-gather around a ring of N simulated ranks whose buffers all live in
// one GPU's memory, under one of three protocols (LL, LL128, Simple); the
// same ring runs ReduceScatter and AllGather alone.  Also here: the direct
// (two-shot) algorithm, which reads every rank's segment and writes the sum
// to every rank with no FIFOs, and the streaming copy of the one-rank case.
//
// Work decomposition.  Grid = nchannels * nranks workgroups; workgroup
// (channel c, rank r) holds `nwaves` wavefronts and each wavefront is an
// independent ring member: wave w of rank r talks only to wave w of ranks
// r-1 and r+1 of the same channel, through its own FIFO slots and its own
// head/tail counters, so no wave ever waits on a workgroup barrier.
//
// Segment-major schedule (the same order the oracle follows).  Element
// ranges: seg = roundup(ceil(count/N), A) per segment, then a channel's
// sub-range of cs elements, then chunk steps of `chunk` elements, of which
// wave w takes kw elements.  For every chunk step j, rank r runs ring steps
// k = 0 .. 2N-2 on segment s = (r - k) mod N:
//   k = 0         send its own input           (reduce-scatter start)
//   0 < k < N-1   recv + own input -> send      (recvReduceSend)
//   k = N-1       recv + own input -> y; write y, send y  (recvReduceCopySend)
//   N-1 < k < 2N-2  recv y; write y, send y     (recvCopySend)
//   k = 2N-2      recv y; write y               (recvCopy)
// so segment s is summed x_s + x_{s+1} + ... + x_{s+N-1} in that order.  In
// the peer-direct mode step 0 becomes a read of the chain start's input by
// the second rank, and the Simple ring writes all-gather chunks into the
// next rank's output instead of a FIFO slot.
//
// Memory model.  A FIFO slot written by one wave is read by a wave that can
// sit on another XCD, i.e. behind another L2.  Every FIFO access therefore
// uses the device-scope coherence bit (sc1) -- the same encoding the
// compiler uses for device-scope atomic loads and stores on this target --
// and every counter is a device-scope atomic.  A Simple or LL128 sender
// makes its data writes complete (s_waitcnt vmcnt(0)) before it stores the
// counter or flags that publish them; an LL line carries its own flag.  A
// Simple receiver issues its slot reads only after it has observed the
// counter; LL and LL128 receivers read data and flags together and accept a
// line once its flag is current (for LL128 see the note at LL128Step).  Rank
// inputs are read with the non-temporal hint: nothing writes an
// input before every read of it.  Rank outputs are written non-temporally
// by their own rank, except in the peer-direct mode, where a neighbour on
// another XCD also writes them, so every output access there uses sc1.
//
// Every wait is bounded by a watchdog on the 100 MHz real-time counter; a
// wave that times out raises the plan's abort word and status bit, and all
// waves leave their loops when they see the abort word, so the kernel always
// drains.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ar_internal.h"

namespace ar {
namespace dev {

typedef uint32_t u32x4 __attribute__((__vector_size__(16)));
typedef uint32_t u32x2 __attribute__((__vector_size__(8)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

// Cache-policy operand of gfx950 buffer instructions.
enum : int { kPolPlain = 0, kPolSc0 = 1, kPolNt = 2, kPolSc1 = 16 };
// The policies are fixed, not build options.  A FIFO line (or, in the
// peer-direct mode, an output element) is written on one XCD and read on
// another, behind a different L2; without the device-scope bit on both the
// write and the read, a reader can be served a stale copy and the ring
// returns wrong sums or waits until the watchdog fires.
constexpr int kFifoLd = kPolSc1;  // device-coherent FIFO reads
constexpr int kFifoSt = kPolSc1;  // device-coherent FIFO writes
constexpr int kInPol = kPolNt;    // rank inputs: read once, streamed
constexpr int kOutPol = kPolNt;   // rank outputs: written once, streamed
static_assert((kFifoLd & kPolSc1) != 0 && (kFifoSt & kPolSc1) != 0, "FIFO accesses must be device-coherent");

enum Kind : int {
    kSend = 0,            // own input -> wire (reduce-scatter start)
    kRecvReduceSend,      // wire + own input -> wire
    kRecvReduceCopySend,  // wire + own input -> output and wire (AllReduce owner)
    kRecvCopySend,        // wire -> output and wire
    kRecvCopy,            // wire -> output
    kRecvReduceCopy,      // wire + own input -> output (ReduceScatter owner)
    kCopySend,            // own input -> output and wire (AllGather start)
    // Simple peer-direct mode: the chain's second rank reads the chain start's
    // input straight from that rank's buffer instead of a first FIFO hop.
    kPeerReduceSend,      // peer input + own input -> wire
    kPeerReduceCopySend,  // peer input + own input -> output and wire (2-rank AllReduce owner)
    kPeerReduceCopy       // peer input + own input -> output (2-rank ReduceScatter owner)
};

// What a step kind does, shared by the three protocols.
template <int KIND>
struct KindTraits {
    static constexpr bool kRecvRS = KIND == kRecvReduceSend || KIND == kRecvReduceCopySend || KIND == kRecvReduceCopy;
    static constexpr bool kRecvAG = KIND == kRecvCopySend || KIND == kRecvCopy;
    // the partial to add is the chain start's input, read from its buffer
    static constexpr bool kRecvPeer = KIND == kPeerReduceSend || KIND == kPeerReduceCopySend || KIND == kPeerReduceCopy;
    static constexpr bool kLoadIn = KIND == kSend || kRecvRS || KIND == kCopySend || kRecvPeer;
    static constexpr bool kSendRS = KIND == kSend || KIND == kRecvReduceSend || KIND == kPeerReduceSend;
    static constexpr bool kSendAG = KIND == kRecvReduceCopySend || KIND == kRecvCopySend || KIND == kCopySend ||
                                    KIND == kPeerReduceCopySend;
    static constexpr bool kReduceToY = KIND == kRecvReduceCopySend || KIND == kRecvReduceCopy ||
                                       KIND == kPeerReduceCopySend || KIND == kPeerReduceCopy;  // y = rounded sum
    static constexpr bool kWriteOut = kReduceToY || kRecvAG || KIND == kCopySend;
    static constexpr bool kCopyInToY = KIND == kCopySend;                                      // y = own input
};

template <int DT> struct Elem;
template <> struct Elem<AR_FLOAT32> { static constexpr uint32_t E = 4, A = 4; };
template <> struct Elem<AR_BFLOAT16> { static constexpr uint32_t E = 2, A = 8; };

__device__ __forceinline__ Rsrc make_rsrc(const void *p, uint64_t bytes)
{
    // Word 3 = 0x00020000: raw 32-bit dword format, as on the rest of CDNA.
    uint32_t n = bytes > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)n, 0x00020000);
}

template <int POL> __device__ __forceinline__ u32x4 ld128(Rsrc r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ u32x2 ld64(Rsrc r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ uint32_t ld32(Rsrc r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ uint32_t ld16(Rsrc r, uint32_t off)
{
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ void st128(Rsrc r, uint32_t off, u32x4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ void st64(Rsrc r, uint32_t off, u32x2 v)
{
    __builtin_amdgcn_raw_buffer_store_b64(v, r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ void st32(Rsrc r, uint32_t off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, POL);
}
template <int POL> __device__ __forceinline__ void st16(Rsrc r, uint32_t off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)v, r, (int)off, 0, POL);
}

// A buffer offset outside every resource built by the ring steps (each covers
// at most one step's data or one FIFO slot, far below 2^31 bytes): a load
// there returns zeros and a store there is dropped, by the hardware's range
// check.  Lanes past the end of a message use it instead of a branch, which
// keeps a batch of accesses straight-line code; the compiler can then wait
// for exactly the loads an instruction needs instead of for every
// outstanding access (a branch around each access makes it wait for all of
// them, earlier stores included, before each store).
constexpr uint32_t kOobOff = 0x80000000u;
__device__ __forceinline__ uint32_t in_range(bool ok, uint32_t off) { return ok ? off : kOobOff; }

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & 63u; }

// True on every lane when p holds on any active lane; the result is a
// wave-uniform value the compiler knows to be uniform.
//
// Uniformity matters throughout the ring steps: a branch on the lane (such as
// "lane 0 stores the flag") whose join merges any value makes the compiler
// treat everything that depends on it as per-lane.  The step loop then runs
// under an execution mask, loop-carried counters and pointers move into
// vector registers, and every buffer access is wrapped in a loop that reads
// its descriptor lane by lane.  So flags are stored by every lane (the same
// value to the same address: one write), and partial units and groups use
// out-of-range offsets instead of lane branches.
__device__ __forceinline__ bool any_lane(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0; }

// The lane index as a value the compiler may not hoist out of the step loop:
// a step's per-lane offsets are then recomputed each step (a few ALU ops)
// instead of being held in registers across every step of the kernel.
__device__ __forceinline__ uint32_t step_lane()
{
    uint32_t l = lane_id();
    asm volatile("" : "+v"(l));
    return l;
}

__device__ __forceinline__ uint64_t uniform64(uint64_t v)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// ---- fp32 / bf16 ------------------------------------------------------------

__device__ __forceinline__ float as_f32(uint32_t u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ uint32_t as_u32(float f) { return __builtin_bit_cast(uint32_t, f); }

// bf16 -> fp32 is exact: the bf16 bits are the top half of the fp32 word.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return as_f32(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return as_f32(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest even; NaN -> quiet NaN 0x7FC0.
__device__ __forceinline__ uint32_t bf16_rne(float f)
{
    uint32_t u = as_u32(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return bf16_rne(lo) | (bf16_rne(hi) << 16);
}

// ---- flags, fences, watchdog ----------------------------------------------

__device__ __forceinline__ uint64_t flag_load(const uint64_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void flag_store(uint64_t *p, uint64_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Make every earlier memory operation of this wave complete before what
// follows is issued: s_waitcnt vmcnt(0) (expcnt and lgkmcnt left alone),
// with compiler fences on both sides so no access is moved across it.
__device__ __forceinline__ void drain_vmem()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Keep later loads behind an observed flag (compiler ordering; the hardware
// issues them after the flag value has been tested).
__device__ __forceinline__ void after_observe() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup"); }

struct Watchdog {
    uint64_t start = 0;
    uint32_t iter = 0;
};

// Returns true when the wave must give up: another wave aborted, or this
// wait has exceeded the timeout (then this wave raises the abort itself).
__device__ __forceinline__ bool watchdog_expired(const RingArgs &a, Watchdog &wd)
{
    if ((++wd.iter & 31u) != 0) return false;
    uint32_t ab = __hip_atomic_load(a.ctl + kCtlAbort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (__builtin_amdgcn_readfirstlane(ab) != 0) return true;
    uint64_t now = uniform64(wall_clock64());
    if (wd.start == 0) {
        wd.start = now;
        return false;
    }
    if (now - wd.start > a.timeout_ticks) {
        {  // every lane (see any_lane): the same bit, the same word
            __hip_atomic_fetch_or(a.ctl + kCtlStatus, kStatusTimeout, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.ctl + kCtlAbort, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        return true;
    }
    return false;
}

// Wait until *flag >= target.  `cache` holds the last value seen.
__device__ __forceinline__ bool wait_geq(const RingArgs &a, const uint64_t *flag, uint64_t target,
                                         uint64_t &cache)
{
    if (cache >= target) return true;
    Watchdog wd;
    while (true) {
        uint64_t v = uniform64(flag_load(flag));
        if (v >= target) {
            cache = v;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
        if (watchdog_expired(a, wd)) return false;
    }
    after_observe();
    return true;
}

// Wait until *f1 >= t1 and, when f2 is given, *f2 >= t2, reading both
// counters in each round trip (a receiver's incoming tail and its outgoing
// head: the send credit then costs no round trip of its own).
__device__ __forceinline__ bool wait_geq2(const RingArgs &a, const uint64_t *f1, uint64_t t1, uint64_t &c1,
                                          const uint64_t *f2, uint64_t t2, uint64_t &c2)
{
    const bool two = f2 != nullptr;
    if (c1 >= t1 && (!two || c2 >= t2)) return true;
    const uint64_t *g2 = two ? f2 : f1;
    Watchdog wd;
    while (true) {
        const uint64_t v1 = uniform64(flag_load(f1));
        const uint64_t v2 = uniform64(flag_load(g2));
        if (v1 > c1) c1 = v1;
        if (two && v2 > c2) c2 = v2;
        if (c1 >= t1 && (!two || c2 >= t2)) break;
        __builtin_amdgcn_s_sleep(1);
        if (watchdog_expired(a, wd)) return false;
    }
    after_observe();
    return true;
}

__device__ __forceinline__ void debug_jitter(const RingArgs &a, uint64_t salt)
{
    if (!(a.debug & AR_DEBUG_JITTER)) return;
    uint64_t h = salt * 0x9E3779B97F4A7C15ull;
    h ^= h >> 29;
    uint32_t n = (uint32_t)(h & 63u);
    for (uint32_t i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(8);
}

// ---- debug state (kernel builds with the debug hooks only) -----------------

// One step's record of AR_DEBUG_TRACE, stamped with the 100 MHz real-time
// counter (the same clock on every XCD).  Fields, in order:
//   t_begin   step entered
//   t_recv    first data of the step accepted (flag or counter observed)
//   polls     LL: reloads before the first batch was accepted; LL128: 1 if
//             the first look at the first batch was stale; Simple: 0
//   t_issued  the step's (first drain group's) data stores issued
//   t_drained those stores complete (Simple, LL128; LL has no drain: 0)
//   t_posted  the flag / counter that publishes them stored
//   msg       index of the message sent (or, for a receive-only step, taken)
//   kind      the step kind (Kind)
struct StepTrace {
    uint64_t t_begin, t_recv, polls, t_issued, t_drained, t_posted, msg, kind;
};

struct DbgState {
    bool check;            // AR_DEBUG_CHECK_LINES
    bool trace;            // AR_DEBUG_TRACE, and this wave is channel 0 / wave 0
    uint32_t checked;      // lines accepted and checked
    uint32_t first;        // of those, accepted on the first load
    uint32_t bad;          // of those, with data not matching the flag
    uint32_t step;         // steps of this run so far (trace index)
    StepTrace tr;
};

__device__ __forceinline__ uint64_t now_ticks() { return uniform64(wall_clock64()); }

// AR_DEBUG_CHECK_LINES: the data word a writer stores at byte `off` of a
// slot for the message whose 32-bit flag is `tag`.  For a fixed offset it is
// a bijection of the tag (an odd multiplier, then fixed terms), so data left
// by any other message never matches; for a fixed tag it changes with the
// offset, so misplaced data does not match either.
__device__ __forceinline__ uint32_t check_word(uint32_t tag, uint32_t off)
{
    return (tag * 0x9E3779B1u) ^ (off * 0x85EBCA6Bu) ^ 0x5BD1E995u;
}

// Lines with any bit set in an 8-lane group of a 64-lane mask.
__device__ __forceinline__ uint32_t groups8_set(uint64_t m)
{
    m |= m >> 4;
    m |= m >> 2;
    m |= m >> 1;
    return (uint32_t)__builtin_popcountll(m & 0x0101010101010101ull);
}

// ---- per-wave ring state ---------------------------------------------------

struct Ring {
    const RingArgs *a;
    uint32_t N, r, c, w;
    uint64_t *tail_out, *head_out;  // link r -> r+1: I write tail, read head
    uint64_t *tail_in, *head_in;    // link r-1 -> r: I read tail, write head
    char *fifo_out;
    const char *fifo_in;
    uint64_t m_out, m_in;           // absolute index of the next message out / in
    uint64_t head_seen, tail_seen;  // last counter values observed
    uint32_t slot_out, slot_in;     // FIFO slot of message m_out / m_in: m mod depth
    DbgState dbg;                   // used by the builds with the debug hooks only
};

// LL flag of message m: the low 32 bits of m + 1.  A line left in a slot by
// an earlier message carries that message's flag, and a plan keeps every
// stale line fewer than 2^31 messages old (the same per-run message pattern
// repeats, so each line of a slot is rewritten within depth * msgs_per_run
// messages), so a stale flag never equals the current one.  Fresh (zeroed)
// memory is only ever read within the first such window, when flags are
// small and nonzero.
__device__ __forceinline__ uint32_t ll_tag(uint64_t m) { return (uint32_t)m + 1u; }

__device__ __forceinline__ char *slot_ptr(char *base, uint32_t slot, const RingArgs &a)
{
    return base + (uint64_t)slot * a.slot_bytes;
}

// Step to the next message on the outgoing / incoming link (no divisions on
// the per-message path).
__device__ __forceinline__ void advance_out(Ring &g)
{
    ++g.m_out;
    g.slot_out = g.slot_out + 1 == g.a->depth ? 0u : g.slot_out + 1;
}
__device__ __forceinline__ void advance_in(Ring &g)
{
    ++g.m_in;
    g.slot_in = g.slot_in + 1 == g.a->depth ? 0u : g.slot_in + 1;
}

// True when the last head value seen already frees the slot of message
// m_out (the receiver has consumed message m_out - depth).
__device__ __forceinline__ bool slot_free_cached(const Ring &g)
{
    const uint64_t d = g.a->depth;
    return g.m_out + 1 <= d || g.head_seen >= g.m_out + 1 - d;
}

// Sender side: wait until the slot of message m_out is free, i.e. the
// receiver has consumed message m_out - depth.
__device__ __forceinline__ bool acquire_send_slot(Ring &g)
{
    const uint64_t d = g.a->depth;
    if (g.m_out + 1 <= d) return true;  // first `depth` messages of the plan's life
    return wait_geq(*g.a, g.head_out, g.m_out + 1 - d, g.head_seen);
}

// Debug: channel 0 / wave 0 / rank 0 announces none of its messages, so its
// successor waits until the watchdog fires (a monotone counter would let a
// later post cover a single skipped one).
__device__ __forceinline__ bool skip_this_post(const Ring &g)
{
    return (g.a->debug & AR_DEBUG_SKIP_POST) && g.c == 0 && g.w == 0 && g.r == 0;
}

// Byte offset, in a slot, of 16-byte vector v (of `nv` per item) of item i
// when a message holds n items and every item is wider than one vector (the
// fp32 partials of bf16 data).  Items are taken in blocks of 64, one per
// lane, and within a block vector v of every item comes before vector v + 1
// of any: one store instruction of a wave then covers one contiguous stretch
// instead of every other 16 bytes, which would make the device-coherent
// write-through send each 64-byte sector twice.  With nv = 1 this is i * 16.
__device__ __forceinline__ uint32_t wide_off(uint32_t i, uint32_t v, uint32_t nv, uint32_t n)
{
    const uint32_t blk = i & ~63u;
    const uint32_t in_blk = n - blk < 64u ? n - blk : 64u;
    return blk * nv * 16 + v * in_blk * 16 + (i & 63u) * 16;
}

// ===================================================================== Simple
//
// Slot layout: the message's elements as fp32 partials during the
// reduce-scatter (A*4 bytes per unit of A elements, placed by wide_off) and
// in the data type during the all-gather (16 bytes per unit, back to back).
// A unit is A elements = 16 bytes of the data type; lanes take consecutive
// units, U units per lane per batch, all loads of a batch before its stores.
//
// DAG (peer-direct mode) uses the neighbours' buffers where that saves a
// copy.  (1) An all-gather message is not staged in the FIFO: the sender
// writes the finished values straight into the next rank's output buffer, at
// the place they belong, and announces them with the same tail counter; the
// receiver forwards them from its own output buffer, and the last hop of the
// ring moves no data at all.  (2) A reduction chain has no first FIFO hop:
// its second rank reads the chain start's input from that rank's buffer.
// Every access to an output buffer in this mode is device-coherent, because
// ranks on other XCDs write into it.

template <int DT, int KIND, bool DAG>
struct SimpleStep {
    static constexpr uint32_t A = Elem<DT>::A;
    static constexpr uint32_t E = Elem<DT>::E;
    static constexpr uint32_t RSV = A / 4;  // 16-byte fp32 vectors per unit on the RS wire
    static constexpr bool kRecvRS = KindTraits<KIND>::kRecvRS;
    static constexpr bool kRecvAG = KindTraits<KIND>::kRecvAG;
    static constexpr bool kLoadIn = KindTraits<KIND>::kLoadIn;
    static constexpr bool kSendRS = KindTraits<KIND>::kSendRS;
    static constexpr bool kSendAG = KindTraits<KIND>::kSendAG;
    static constexpr bool kWriteOut = KindTraits<KIND>::kWriteOut;
    static constexpr bool kReduceToY = KindTraits<KIND>::kReduceToY;
    static constexpr bool kCopyInToY = KindTraits<KIND>::kCopyInToY;
    static constexpr bool kRecvPeer = KindTraits<KIND>::kRecvPeer;
    static constexpr int U = 4;
    // With DAG a received all-gather message is already in the own output.
    static constexpr bool kWriteOwn = kWriteOut && !(DAG && kRecvAG);
    static constexpr int kOwnPol = DAG ? kFifoSt : kOutPol;  // own output stores
    static constexpr int kAgLdPol = kFifoLd;                  // all-gather reads (FIFO or own output)

    // Partial last unit of the buffer: element-wise data accesses.
    template <int POL>
    __device__ static u32x4 load_partial(Rsrc r, uint32_t off, uint32_t valid)
    {
        u32x4 v = {0, 0, 0, 0};
        if (E == 4) {
            for (uint32_t i = 0; i < valid; ++i) v[i] = ld32<POL>(r, off + 4 * i);
        } else {
            for (uint32_t i = 0; i < valid; ++i) {
                uint32_t h = ld16<POL>(r, off + 2 * i);
                v[i >> 1] |= (i & 1) ? (h << 16) : h;
            }
        }
        return v;
    }
    template <int POL>
    __device__ static void store_partial(Rsrc r, uint32_t off, u32x4 v, uint32_t valid)
    {
        if (E == 4) {
            for (uint32_t i = 0; i < valid; ++i) st32<POL>(r, off + 4 * i, v[i]);
        } else {
            for (uint32_t i = 0; i < valid; ++i) st16<POL>(r, off + 2 * i, (i & 1) ? (v[i >> 1] >> 16) : (v[i >> 1] & 0xFFFFu));
        }
    }

    // acc[A] = RS wire partials (or the widened peer input) + widened input
    // (or just the input at k = 0).
    __device__ static void reduce(const u32x4 *rs, u32x4 in, float *acc)
    {
        if (E == 4) {
            for (int i = 0; i < 4; ++i) acc[i] = as_f32(in[i]);
        } else {
            for (int i = 0; i < 4; ++i) {
                acc[2 * i] = bf16_lo(in[i]);
                acc[2 * i + 1] = bf16_hi(in[i]);
            }
        }
        if (kRecvRS) {
            for (uint32_t v = 0; v < RSV; ++v)
                for (int i = 0; i < 4; ++i) acc[4 * v + i] = as_f32(rs[v][i]) + acc[4 * v + i];
        }
        if (kRecvPeer) {  // rs[0]: the chain start's unit, in the data type
            if (E == 4) {
                for (int i = 0; i < 4; ++i) acc[i] = as_f32(rs[0][i]) + acc[i];
            } else {
                for (int i = 0; i < 4; ++i) {
                    acc[2 * i] = bf16_lo(rs[0][i]) + acc[2 * i];
                    acc[2 * i + 1] = bf16_hi(rs[0][i]) + acc[2 * i + 1];
                }
            }
        }
    }

    // ok = false: a lane past the end of the message, whose full-unit
    // accesses are sent out of range.
    __device__ static void unit(Rsrc rout, Rsrc wo, uint32_t u, bool ok, uint32_t valid, uint32_t nunits,
                                const u32x4 &in, const u32x4 *rs, const u32x4 &ag)
    {
        static_assert(!kRecvPeer || DAG, "peer reads belong to the peer-direct mode");
        float acc[A];
        if (kSendRS || kReduceToY) reduce(rs, in, acc);
        if (kSendRS) {
            for (uint32_t v = 0; v < RSV; ++v) {
                u32x4 o = {as_u32(acc[4 * v]), as_u32(acc[4 * v + 1]), as_u32(acc[4 * v + 2]),
                           as_u32(acc[4 * v + 3])};
                st128<kFifoSt>(wo, in_range(ok, wide_off(u, v, RSV, nunits)), o);
            }
        }
        u32x4 y;
        if (kReduceToY) {
            if (E == 4) {
                y = u32x4{as_u32(acc[0]), as_u32(acc[1]), as_u32(acc[2]), as_u32(acc[3])};
            } else {
                for (int i = 0; i < 4; ++i) y[i] = pack_bf16(acc[2 * i], acc[2 * i + 1]);
            }
        } else if (kCopyInToY) {
            y = in;
        } else {
            y = ag;
        }
        if (kWriteOwn) {
            if (valid == A) st128<kOwnPol>(rout, in_range(ok, u * 16), y);
            else store_partial<kOwnPol>(rout, u * 16, y, valid);
        }
        if (kSendAG) {
            // A FIFO slot is padded to whole units; the next rank's output is not.
            if (valid == A || !DAG) st128<kFifoSt>(wo, in_range(ok, u * 16), y);
            else store_partial<kFifoSt>(wo, u * 16, y, valid);
        }
    }

    // rslot / wslot: FIFO slots, or with DAG for all-gather messages the own
    // and the next rank's output at this message's elements.
    __device__ static void run(const RingArgs &a, const char *src, char *dst, const char *rslot,
                               char *wslot, uint32_t len)
    {
        if (DAG && KIND == kRecvCopy) return;  // the data is already in place (simple_step skips it)
        const uint32_t lane = step_lane();
        const uint32_t nfull = len / A, rem = len % A;
        const uint32_t nunits = nfull + (rem ? 1u : 0u);
        const Rsrc rin = make_rsrc(src, (uint64_t)len * E);
        const Rsrc rout = make_rsrc(dst, (uint64_t)len * E);
        const Rsrc wi = make_rsrc(rslot, (DAG && kRecvAG) || kRecvPeer ? (uint64_t)len * E : a.slot_bytes);
        const Rsrc wo = make_rsrc(wslot, DAG && kSendAG ? (uint64_t)len * E : a.slot_bytes);
        for (uint32_t base = 0; base < nfull; base += 64 * U) {
            u32x4 in[U], rs[U][RSV], ag[U];
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const uint32_t u = base + 64 * t + lane;
                const bool ok = u < nfull;
                if (kLoadIn) in[t] = ld128<kInPol>(rin, in_range(ok, u * 16));
                if (kRecvRS)
                    for (uint32_t v = 0; v < RSV; ++v)
                        rs[t][v] = ld128<kFifoLd>(wi, in_range(ok, wide_off(u, v, RSV, nunits)));
                if (kRecvPeer) rs[t][0] = ld128<kInPol>(wi, in_range(ok, u * 16));
                if (kRecvAG) ag[t] = ld128<kAgLdPol>(wi, in_range(ok, u * 16));
            }
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const uint32_t u = base + 64 * t + lane;
                unit(rout, wo, u, u < nfull, A, nunits, in[t], rs[t], ag[t]);
            }
        }
        if (rem && lane == (nfull & 63u)) {
            const uint32_t u = nfull;
            u32x4 in = {0, 0, 0, 0}, rs[RSV], ag = {0, 0, 0, 0};
            if (kLoadIn) in = load_partial<kInPol>(rin, u * 16, rem);
            if (kRecvRS)
                for (uint32_t v = 0; v < RSV; ++v) rs[v] = ld128<kFifoLd>(wi, wide_off(u, v, RSV, nunits));
            if (kRecvPeer) rs[0] = load_partial<kInPol>(wi, u * 16, rem);
            if (kRecvAG) ag = DAG ? load_partial<kAgLdPol>(wi, u * 16, rem) : ld128<kAgLdPol>(wi, u * 16);
            unit(rout, wo, u, true, rem, nunits, in, rs, ag);
        }
    }
};

// dst: this step's elements in the own output; peer_dst: the same elements
// in the next rank's output (DAG all-gather sends); peer_src: the same
// elements of the previous rank's input (peer-direct chain starts).
template <int DT, int KIND, bool DAG, bool DBG>
__device__ __forceinline__ bool simple_step(Ring &g, const char *src, char *dst, char *peer_dst,
                                            const char *peer_src, uint32_t len)
{
    const RingArgs &a = *g.a;
    if constexpr (DAG && KIND == kRecvCopy) {
        // The last hop of a peer-direct all-gather: the predecessor writes
        // the values straight into this rank's output, and nothing else in
        // this run reads or writes them, so there is nothing to wait for;
        // they are in place when the kernel ends.  The message is
        // acknowledged at once: it occupies no FIFO slot, and every earlier
        // message of the link has been consumed, in order.
        flag_store(g.head_in, g.m_in + 1);
        advance_in(g);
        return true;
    }
    // A peer read needs no message: the chain start's input is in place
    // before the kernel starts and stays there until the chain is done.
    constexpr bool recv = KindTraits<KIND>::kRecvRS || KindTraits<KIND>::kRecvAG;
    constexpr bool send = KindTraits<KIND>::kSendRS || KindTraits<KIND>::kSendAG;
    // With DAG only reduce-scatter messages occupy FIFO slots.
    constexpr bool fifo_in = KindTraits<KIND>::kRecvRS || (KindTraits<KIND>::kRecvAG && !DAG);
    constexpr bool fifo_out = KindTraits<KIND>::kSendRS || (KindTraits<KIND>::kSendAG && !DAG);
    const char *rslot = nullptr;
    char *wslot = nullptr;
    if (recv) {
        // The incoming tail and, if the cached credit does not cover this
        // message, the outgoing head are polled together.
        const bool credit = fifo_out && !slot_free_cached(g);
        if (!wait_geq2(a, g.tail_in, g.m_in + 1, g.tail_seen, credit ? g.head_out : nullptr,
                       g.m_out + 1 - a.depth, g.head_seen))
            return false;
        if constexpr (DBG)
            if (g.dbg.trace) g.dbg.tr.t_recv = now_ticks();
        rslot = fifo_in ? slot_ptr(const_cast<char *>(g.fifo_in), g.slot_in, a) : dst;
    }
    if (KindTraits<KIND>::kRecvPeer) rslot = peer_src;
    if (send) {
        if (fifo_out && !acquire_send_slot(g)) return false;
        wslot = fifo_out ? slot_ptr(g.fifo_out, g.slot_out, a) : peer_dst;
    }
    SimpleStep<DT, KIND, DAG>::run(a, src, dst, rslot, wslot, len);
    if constexpr (DBG)
        if (g.dbg.trace) g.dbg.tr.t_issued = now_ticks();
    // Slot writes (and slot reads) complete before either counter moves.
    drain_vmem();
    if constexpr (DBG)
        if (g.dbg.trace) g.dbg.tr.t_drained = now_ticks();
    if (send) {
        if constexpr (DBG) debug_jitter(a, g.m_out ^ ((uint64_t)g.r << 40) ^ ((uint64_t)g.c << 48));
        if (!(DBG && skip_this_post(g))) flag_store(g.tail_out, g.m_out + 1);
        if constexpr (DBG)
            if (g.dbg.trace) g.dbg.tr.t_posted = now_ticks();
        advance_out(g);
    }
    if (recv) {
        flag_store(g.head_in, g.m_in + 1);
        advance_in(g);
    }
    return true;
}

// ========================================================================= LL
//
// 8-byte lines {u32 data, u32 flag}; flag = ll_tag(message index).  One
// 16-byte store carries two lines, so a lane's 16-byte access is two complete
// lines.  Reduce-scatter lines carry one fp32 partial each; all-gather lines
// carry one fp32 or two bf16 values.  Lanes take "groups" of 8 data bytes (2
// fp32 or 4 bf16): input/output 8 bytes, RS wire G lines (placed by
// wide_off), AG wire 2 lines (16 bytes).  In the peer-direct mode a
// reduction chain starts as in the Simple ring: its second rank reads the
// chain start's input (8 bytes per group, no flags) from that rank's buffer;
// the all-gather keeps its lines, whose flags cannot live in a user buffer.

template <int DT, int KIND, bool DBG>
struct LLStep {
    static constexpr uint32_t E = Elem<DT>::E;
    static constexpr uint32_t G = 8 / E;         // elements per group
    static constexpr uint32_t RSV = G / 2;       // 16-byte wire ops per group on the RS wire
    static constexpr bool kRecvRS = KindTraits<KIND>::kRecvRS;
    static constexpr bool kRecvAG = KindTraits<KIND>::kRecvAG;
    static constexpr bool kLoadIn = KindTraits<KIND>::kLoadIn;
    static constexpr bool kSendRS = KindTraits<KIND>::kSendRS;
    static constexpr bool kSendAG = KindTraits<KIND>::kSendAG;
    static constexpr bool kWriteOut = KindTraits<KIND>::kWriteOut;
    static constexpr bool kReduceToY = KindTraits<KIND>::kReduceToY;
    static constexpr bool kCopyInToY = KindTraits<KIND>::kCopyInToY;
    static constexpr bool kRecvPeer = KindTraits<KIND>::kRecvPeer;
    static constexpr int U = 4;

    // A partial group (valid < G elements) moves element by element; ok =
    // false sends every access out of range.
    __device__ static u32x2 load_part(Rsrc r, uint32_t q, uint32_t valid, bool ok)
    {
        u32x2 v = {0, 0};
        for (uint32_t i = 0; i < valid; ++i) {
            if (E == 4) v[i] = ld32<kInPol>(r, in_range(ok, q * 8 + 4 * i));
            else v[i >> 1] |= ld16<kInPol>(r, in_range(ok, q * 8 + 2 * i)) << ((i & 1) * 16);
        }
        return v;
    }
    __device__ static void store_part(Rsrc r, uint32_t q, u32x2 v, uint32_t valid, bool ok)
    {
        for (uint32_t i = 0; i < valid; ++i) {
            if (E == 4) st32<kOutPol>(r, in_range(ok, q * 8 + 4 * i), v[i]);
            else st16<kOutPol>(r, in_range(ok, q * 8 + 2 * i), (v[i >> 1] >> ((i & 1) * 16)) & 0xFFFFu);
        }
    }

    __device__ static bool lines_ok(const u32x4 &l, uint32_t tag) { return l[1] == tag && l[3] == tag; }

    // One group's arithmetic and stores; ok = false sends every access out
    // of range (a lane past the end of the message).  chk (debug builds
    // only): the wire carries check words instead of data.
    __device__ static void group(Rsrc rout, Rsrc wo, uint32_t q, bool ok, uint32_t valid, uint32_t ng,
                                 u32x2 in, const u32x4 *rs, const u32x4 &ag, u32x2 pe, uint32_t tag_out, bool chk)
    {
        float acc[G];
        if (kSendRS || kReduceToY) {
            if (E == 4) {
                acc[0] = as_f32(in[0]);
                acc[1] = as_f32(in[1]);
            } else {
                acc[0] = bf16_lo(in[0]);
                acc[1] = bf16_hi(in[0]);
                acc[2] = bf16_lo(in[1]);
                acc[3] = bf16_hi(in[1]);
            }
            if (kRecvRS) {
                for (uint32_t v = 0; v < RSV; ++v) {
                    acc[2 * v] = as_f32(rs[v][0]) + acc[2 * v];
                    acc[2 * v + 1] = as_f32(rs[v][2]) + acc[2 * v + 1];
                }
            }
            if (kRecvPeer) {  // the chain start's elements, in the data type
                if (E == 4) {
                    acc[0] = as_f32(pe[0]) + acc[0];
                    acc[1] = as_f32(pe[1]) + acc[1];
                } else {
                    acc[0] = bf16_lo(pe[0]) + acc[0];
                    acc[1] = bf16_hi(pe[0]) + acc[1];
                    acc[2] = bf16_lo(pe[1]) + acc[2];
                    acc[3] = bf16_hi(pe[1]) + acc[3];
                }
            }
        }
        if (kSendRS) {
            for (uint32_t v = 0; v < RSV; ++v) {
                const uint32_t off = wide_off(q, v, RSV, ng);
                u32x4 o = {as_u32(acc[2 * v]), tag_out, as_u32(acc[2 * v + 1]), tag_out};
                if (DBG && chk) o = u32x4{check_word(tag_out, off), tag_out, check_word(tag_out, off + 8), tag_out};
                st128<kFifoSt>(wo, in_range(ok, off), o);
            }
        }
        u32x2 y;
        if (kReduceToY) {
            if (E == 4) y = u32x2{as_u32(acc[0]), as_u32(acc[1])};
            else y = u32x2{pack_bf16(acc[0], acc[1]), pack_bf16(acc[2], acc[3])};
        } else if (kCopyInToY) {
            y = in;
        } else {
            y = u32x2{ag[0], ag[2]};
        }
        if (kWriteOut) {
            if (valid == G) st64<kOutPol>(rout, in_range(ok, q * 8), y);
            else store_part(rout, q, y, valid, ok);
        }
        if (kSendAG) {
            u32x4 o = {y[0], tag_out, y[1], tag_out};
            if (DBG && chk) o = u32x4{check_word(tag_out, q * 16), tag_out, check_word(tag_out, q * 16 + 8), tag_out};
            st128<kFifoSt>(wo, in_range(ok, q * 16), o);
        }
    }

    // Debug builds: check the data words of the lines a lane accepted (two
    // lines per 16-byte access) against the writer's check words.
    __device__ static void check_access(const u32x4 &l, uint32_t off, bool ok, uint32_t tag, uint32_t first,
                                        DbgState *dbg)
    {
        const bool bad0 = ok && l[0] != check_word(tag, off);
        const bool bad1 = ok && l[2] != check_word(tag, off + 8);
        const uint32_t n = 2 * (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(ok));
        dbg->checked += n;
        dbg->first += first ? n : 0u;
        dbg->bad += (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(bad0)) +
                    (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(bad1));
    }

    // Full groups go in batches of U per lane as straight-line code (lanes
    // past the end use out-of-range offsets); a partial last group is done
    // afterwards by one lane, with its own poll.
    __device__ static bool run(const RingArgs &a, const char *src, char *dst, const char *rslot,
                               char *wslot, uint32_t len, uint32_t tag_in, uint32_t tag_out, DbgState *dbg)
    {
        const uint32_t lane = step_lane();
        const bool chk = DBG && dbg->check;
        const uint32_t nfg = len / G, rem = len % G;
        const uint32_t ng = nfg + (rem ? 1u : 0u);
        const Rsrc rin = make_rsrc(src, (uint64_t)len * E);
        const Rsrc rout = make_rsrc(dst, (uint64_t)len * E);
        // rslot: the incoming FIFO slot, or for a peer read the chain
        // start's input at this message's elements
        const Rsrc wi = make_rsrc(rslot, kRecvPeer ? (uint64_t)len * E : a.slot_bytes);
        const Rsrc wo = make_rsrc(wslot, a.slot_bytes);
        for (uint32_t base = 0; base < nfg; base += 64 * U) {
            u32x2 in[U], pe[U];
            u32x4 rs[U][RSV], ag[U];
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const uint32_t q = base + 64 * t + lane;
                const bool ok = q < nfg;
                if (kLoadIn) in[t] = ld64<kInPol>(rin, in_range(ok, q * 8));
                if (kRecvPeer) pe[t] = ld64<kInPol>(wi, in_range(ok, q * 8));
                if (kRecvRS)
                    for (uint32_t v = 0; v < RSV; ++v)
                        rs[t][v] = ld128<kFifoLd>(wi, in_range(ok, wide_off(q, v, RSV, ng)));
                if (kRecvAG) ag[t] = ld128<kFifoLd>(wi, in_range(ok, q * 16));
            }
            if (kRecvRS || kRecvAG) {
                // Spin until every line this wave needs carries the expected
                // flag, reloading all of them each time (a line that is
                // already valid cannot change before this wave frees the slot).
                Watchdog wd;
                uint32_t reloads = 0;
                while (true) {
                    bool bad = false;
#pragma unroll
                    for (int t = 0; t < U; ++t) {
                        const bool ok = base + 64 * t + lane < nfg;
                        if (kRecvRS)
                            for (uint32_t v = 0; v < RSV; ++v) bad |= ok && !lines_ok(rs[t][v], tag_in);
                        if (kRecvAG) bad |= ok && !lines_ok(ag[t], tag_in);
                    }
                    if (!any_lane(bad)) break;
                    __builtin_amdgcn_s_sleep(1);
                    if (watchdog_expired(a, wd)) return false;
                    ++reloads;
#pragma unroll
                    for (int t = 0; t < U; ++t) {
                        const uint32_t q = base + 64 * t + lane;
                        const bool ok = q < nfg;
                        if (kRecvRS)
                            for (uint32_t v = 0; v < RSV; ++v)
                                rs[t][v] = ld128<kFifoLd>(wi, in_range(ok, wide_off(q, v, RSV, ng)));
                        if (kRecvAG) ag[t] = ld128<kFifoLd>(wi, in_range(ok, q * 16));
                    }
                }
                if constexpr (DBG) {
                    if (dbg->trace && dbg->tr.t_recv == 0) {
                        dbg->tr.t_recv = now_ticks();
                        dbg->tr.polls = reloads;
                    }
                    if (chk) {
#pragma unroll
                        for (int t = 0; t < U; ++t) {
                            const uint32_t q = base + 64 * t + lane;
                            const bool ok = q < nfg;
                            if (kRecvRS)
                                for (uint32_t v = 0; v < RSV; ++v)
                                    check_access(rs[t][v], wide_off(q, v, RSV, ng), ok, tag_in, reloads == 0, dbg);
                            if (kRecvAG) check_access(ag[t], q * 16, ok, tag_in, reloads == 0, dbg);
                        }
                    }
                }
            }
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const uint32_t q = base + 64 * t + lane;
                group(rout, wo, q, q < nfg, G, ng, in[t], rs[t], ag[t], kRecvPeer ? pe[t] : u32x2{0, 0}, tag_out,
                      chk);
            }
        }
        if (rem) {
            // The whole wave runs this (no branch on the lane); only the lane
            // of the partial group has its accesses in range.
            const uint32_t q = nfg;
            const bool me = lane == (nfg & 63u);
            u32x2 in = {0, 0}, pe = {0, 0};
            u32x4 rs[RSV], ag = {0, 0, 0, 0};
            if (kLoadIn) in = load_part(rin, q, rem, me);
            if (kRecvPeer) pe = load_part(wi, q, rem, me);
            if (kRecvRS || kRecvAG) {
                Watchdog wd;
                uint32_t reloads = 0;
                while (true) {
                    bool bad = false;
                    if (kRecvRS)
                        for (uint32_t v = 0; v < RSV; ++v) {
                            rs[v] = ld128<kFifoLd>(wi, in_range(me, wide_off(q, v, RSV, ng)));
                            bad |= me && !lines_ok(rs[v], tag_in);
                        }
                    if (kRecvAG) {
                        ag = ld128<kFifoLd>(wi, in_range(me, q * 16));
                        bad |= me && !lines_ok(ag, tag_in);
                    }
                    if (!any_lane(bad)) break;
                    __builtin_amdgcn_s_sleep(1);
                    if (watchdog_expired(a, wd)) return false;
                    ++reloads;
                }
                if constexpr (DBG) {
                    if (dbg->trace && dbg->tr.t_recv == 0) {
                        dbg->tr.t_recv = now_ticks();
                        dbg->tr.polls = reloads;
                    }
                    if (chk) {
                        if (kRecvRS)
                            for (uint32_t v = 0; v < RSV; ++v)
                                check_access(rs[v], wide_off(q, v, RSV, ng), me, tag_in, reloads == 0, dbg);
                        if (kRecvAG) check_access(ag, q * 16, me, tag_in, reloads == 0, dbg);
                    }
                }
            }
            group(rout, wo, q, me, rem, ng, in, rs, ag, pe, tag_out, chk);
        }
        return true;
    }
};

// peer_src: the chain start's input at this step's elements (peer reads).
template <int DT, int KIND, bool DBG>
__device__ __forceinline__ bool ll_step(Ring &g, const char *src, char *dst, const char *peer_src, uint32_t len)
{
    const RingArgs &a = *g.a;
    constexpr bool recv = KindTraits<KIND>::kRecvRS || KindTraits<KIND>::kRecvAG;
    constexpr bool send = KindTraits<KIND>::kSendRS || KindTraits<KIND>::kSendAG;
    const char *rslot = nullptr;
    char *wslot = nullptr;
    if (recv) rslot = slot_ptr(const_cast<char *>(g.fifo_in), g.slot_in, a);
    if (KindTraits<KIND>::kRecvPeer) rslot = peer_src;
    if (send) {
        if (!acquire_send_slot(g)) return false;
        wslot = slot_ptr(g.fifo_out, g.slot_out, a);
    }
    if constexpr (DBG)
        if (send) debug_jitter(a, g.m_out ^ ((uint64_t)g.r << 40) ^ ((uint64_t)g.c << 48));
    // A skipped post writes the lines with the previous message's flag, which
    // the receiver never accepts for this message.
    const bool skip = DBG && send && skip_this_post(g);
    const uint32_t tag_out = ll_tag(skip ? g.m_out - 1 : g.m_out);
    if (!LLStep<DT, KIND, DBG>::run(a, src, dst, rslot, wslot, len, ll_tag(g.m_in), tag_out, &g.dbg)) return false;
    if constexpr (DBG)
        if (g.dbg.trace) g.dbg.tr.t_issued = g.dbg.tr.t_posted = now_ticks();
    if (send) advance_out(g);
    if (recv) {
        // Every line of the message has been loaded and its flag checked, so
        // no read of the slot is outstanding: free it at once, without
        // waiting for this step's own stores (compiler ordering only).
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        flag_store(g.head_in, g.m_in + 1);
        advance_in(g);
    }
    return true;
}

// ====================================================================== LL128
//
// 128-byte lines: bytes 0..119 data, 120..127 a 64-bit flag (message index
// + 1).  Eight lanes own one line: lanes p = 0..6 move 16 data bytes each,
// lane 7 the last 8 data bytes (and, on a read, the flag).  A wave moves 8
// lines per instruction.  The writer stores the data of a group of lines,
// waits for those stores to complete, then stores the lines' flags, one
// line per lane; the reader loads whole lines and accepts a batch once every
// line's flag matches.  Data and flag of a line then come from one load;
// that the data half of such a load is no older than its flag half is an
// assumption (CDNA does not promise 128-byte single-copy atomicity), not a
// guarantee.  A batch found stale is read again only after its flags alone
// have been seen current, which orders that read after them; plans with
// AR_PLAN_LL128_ORDERED treat every batch that way.
//
// Lane 7's part is half as wide as the others.  Rather than a second, narrow
// access for it (a whole extra instruction for one lane in eight), lane 7
// makes the same full-width access half a part earlier: a load keeps the
// upper half, a store sends lane 6's upper half (taken over by a lane move)
// in front of its own, so lanes 6 and 7 write those bytes with equal values.
// Reduce-scatter lines hold 30 fp32 partials; all-gather lines hold 30 fp32
// or 60 bf16 values.  A bf16 recvReduceCopySend re-lays its results from the
// 30-per-line to the 60-per-line format through LDS.  In the peer-direct
// mode a chain's second rank reads the chain start's input (no flags) in
// the layout of its own input.

constexpr uint32_t kLL128Data = 120;

// LU: 16-byte accesses per lane and batch (8 lines each per wave), chosen
// per plan: 2 when a wave's message spans at most one such batch (16
// lines: fewer instructions and registers per step, which decides a
// latency-bound hop), 4 for longer messages (more lines in flight per
// wait: 9-27 % less time from 64 KiB to 32 MiB per rank at 8 ranks).
template <int DT, int KIND, bool DBG, int LU, bool ORD>
struct LL128Step {
    static constexpr uint32_t E = Elem<DT>::E;
    static constexpr bool kRecvRS = KindTraits<KIND>::kRecvRS;
    static constexpr bool kRecvAG = KindTraits<KIND>::kRecvAG;
    static constexpr bool kLoadIn = KindTraits<KIND>::kLoadIn;
    static constexpr bool kSendRS = KindTraits<KIND>::kSendRS;
    static constexpr bool kSendAG = KindTraits<KIND>::kSendAG;
    static constexpr bool kWriteOut = KindTraits<KIND>::kWriteOut;
    static constexpr bool kReduceToY = KindTraits<KIND>::kReduceToY;
    static constexpr bool kCopyInToY = KindTraits<KIND>::kCopyInToY;
    static constexpr bool kRecvPeer = KindTraits<KIND>::kRecvPeer;
    // bf16 recvReduceCopySend changes the line format on the way through.
    static constexpr bool kRelayout = DT == AR_BFLOAT16 && KIND == kRecvReduceCopySend;
    // Wave-wide line accesses (8 lines each) per batch.  Two batches are in
    // flight: the next one's loads go out before this one's stores.
    static constexpr int U = LU;
    // Batches per drain-and-flag group.
    static constexpr uint32_t kGroup = 8;

    // Elements per line on the wire this step reads / writes.
    static constexpr uint32_t kEplRS = kLL128Data / 4;  // 30 fp32 partials
    static constexpr uint32_t kEplAG = kLL128Data / E;  // 30 fp32 or 60 bf16

    // Lane 6's value, read by lane 7 (lanes 8k+6 and 8k+7 share a DPP row).
    __device__ static uint32_t from_lane_below(uint32_t x)
    {
        return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x111 /* row_shr:1 */, 0xF, 0xF, true);
    }
    // A full-width access (WB bytes) that starts half a part early carries
    // lane 7's part in its upper half.
    template <uint32_t WB>
    __device__ static u32x4 upper_half(const u32x4 &v)
    {
        static_assert(WB == 16 || WB == 8, "lane parts are 16 or 8 bytes");
        if constexpr (WB == 16) return u32x4{v[2], v[3], 0, 0};
        else return u32x4{v[1], 0, 0, 0};
    }
    // What lane 7 stores for that access: lane 6's upper half, then its own part.
    template <uint32_t WB>
    __device__ static u32x4 lane7_word(const u32x4 &v)
    {
        static_assert(WB == 16 || WB == 8, "lane parts are 16 or 8 bytes");
        if constexpr (WB == 16) return u32x4{from_lane_below(v[2]), from_lane_below(v[3]), v[0], v[1]};
        else return u32x4{from_lane_below(v[1]), v[0], 0, 0};
    }

    // Accesses of exactly BYTES (16, 8 or 4) bytes: a lane part of a line is
    // 16 data bytes for lanes 0..6 and 8 for lane 7, in the wire format; the
    // matching part of a rank buffer is part_elems elements of the data type.
    template <uint32_t BYTES, int POL>
    __device__ static u32x4 ld_bytes(Rsrc r, uint32_t off)
    {
        if constexpr (BYTES == 16) {
            return ld128<POL>(r, off);
        } else if constexpr (BYTES == 8) {
            const u32x2 h = ld64<POL>(r, off);
            return u32x4{h[0], h[1], 0, 0};
        } else {
            return u32x4{ld32<POL>(r, off), 0, 0, 0};
        }
    }
    template <uint32_t BYTES, int POL>
    __device__ static void st_bytes(Rsrc r, uint32_t off, u32x4 v)
    {
        if constexpr (BYTES == 16) st128<POL>(r, off, v);
        else if constexpr (BYTES == 8) st64<POL>(r, off, u32x2{v[0], v[1]});
        else st32<POL>(r, off, v[0]);
    }

    // One lane's part of a rank buffer: `full` elements (EPART for lanes
    // 0..6, half of that for lane 7) of which the first n exist.  Every
    // access is issued by every lane, out of range where it does not apply,
    // so no store waits on a branch.
    //
    // Loading takes two calls.  load_whole issues the one full-width access
    // of a whole part (lane 7's starting half a part early) and leaves the
    // loaded words untouched: any arithmetic on them would make the wave wait
    // for this load before it issues the next, and a batch's loads would go
    // out one round trip apart.  part_value, called once the batch has
    // arrived, moves lane 7's half into place and fetches a part cut by the
    // end of the message (at most one per message) element by element,
    // behind a wave-uniform test.
    template <uint32_t EPART>
    __device__ static u32x4 load_whole(Rsrc r, uint32_t off, uint32_t p, uint32_t n, uint32_t full)
    {
        constexpr uint32_t WB = EPART * E;
        const bool whole = n != 0 && n == full;
        return ld_bytes<WB, kInPol>(r, in_range(whole, p == 7 ? off - WB / 2 : off));
    }
    template <uint32_t EPART>
    __device__ static u32x4 part_value(Rsrc r, uint32_t off, uint32_t p, uint32_t n, uint32_t full, const u32x4 &w)
    {
        constexpr uint32_t WB = EPART * E;
        u32x4 v = p == 7 ? upper_half<WB>(w) : w;
        const bool cut = n != 0 && n < full;
        if (any_lane(cut)) {
#pragma unroll
            for (uint32_t i = 0; i < EPART; ++i) {
                const bool ok = cut && i < n;
                if (E == 4) v[i] |= ld32<kInPol>(r, in_range(ok, off + 4 * i));
                else v[i >> 1] |= ld16<kInPol>(r, in_range(ok, off + 2 * i)) << ((i & 1) * 16);
            }
        }
        return v;
    }
    template <uint32_t EPART>
    __device__ static void store_part(Rsrc r, uint32_t off, u32x4 v, uint32_t p, uint32_t n, uint32_t full)
    {
        constexpr uint32_t WB = EPART * E;
        const bool whole = n != 0 && n == full;
        // Lane 7 is whole only if lane 6 is, so the bytes it takes over exist.
        const u32x4 l7 = lane7_word<WB>(v);
        st_bytes<WB, kOutPol>(r, in_range(whole, p == 7 ? off - WB / 2 : off), p == 7 ? l7 : v);
        const bool cut = n != 0 && n < full;
        if (any_lane(cut)) {
#pragma unroll
            for (uint32_t i = 0; i < EPART; ++i) {
                const bool ok = cut && i < n;
                if (E == 4) st32<kOutPol>(r, in_range(ok, off + 4 * i), v[i]);
                else st16<kOutPol>(r, in_range(ok, off + 2 * i), (v[i >> 1] >> ((i & 1) * 16)) & 0xFFFFu);
            }
        }
    }

    // One lane's part of a line on the wire (data only; the flag comes
    // later); act = false sends the store out of range.  Lane 7 writes bytes
    // 104..119, the first 8 of them equal to lane 6's.
    __device__ static void put_data(Rsrc wo, uint32_t line, uint32_t p, bool act, u32x4 d)
    {
        const u32x4 l7 = lane7_word<16>(d);
        st128<kFifoSt>(wo, in_range(act, line * 128 + (p == 7 ? 104u : 16 * p)), p == 7 ? l7 : d);
    }
    // Flags of lines [lo, hi), one line per lane.
    __device__ static void put_flags(Rsrc wo, uint32_t lo, uint32_t hi, uint32_t lane, uint64_t tag)
    {
        for (uint32_t lb = lo; lb < hi; lb += 64) {
            const uint32_t line = lb + lane;
            st64<kFifoSt>(wo, in_range(line < hi, line * 128 + 120), u32x2{(uint32_t)tag, (uint32_t)(tag >> 32)});
        }
    }

    // Reduce-scatter arithmetic for one lane part: up to 4 fp32 partials
    // (or, for a peer read, the chain start's 4 elements in the data type)
    // plus the lane's input elements.
    __device__ static u32x4 rs_reduce(const u32x4 &wire, const u32x4 &in)
    {
        float acc[4];
        for (int i = 0; i < 4; ++i) {
            if (E == 4) acc[i] = as_f32(in[i]);
            else acc[i] = (i & 1) ? bf16_hi(in[i >> 1]) : bf16_lo(in[i >> 1]);
        }
        if (kRecvRS)
            for (int i = 0; i < 4; ++i) acc[i] = as_f32(wire[i]) + acc[i];
        if (kRecvPeer) {
            for (int i = 0; i < 4; ++i) {
                const float w = E == 4 ? as_f32(wire[i]) : ((i & 1) ? bf16_hi(wire[i >> 1]) : bf16_lo(wire[i >> 1]));
                acc[i] = w + acc[i];
            }
        }
        return u32x4{as_u32(acc[0]), as_u32(acc[1]), as_u32(acc[2]), as_u32(acc[3])};
    }
    // A two-rank chain's owner in bf16 (peer read, no reduce-scatter line):
    // 8 elements per lane part in the all-gather format, the chain start's
    // plus the own, rounded once.
    __device__ static u32x4 peer_y8(const u32x4 &peer, const u32x4 &in)
    {
        u32x4 y;
        for (int i = 0; i < 4; ++i)
            y[i] = pack_bf16(bf16_lo(peer[i]) + bf16_lo(in[i]), bf16_hi(peer[i]) + bf16_hi(in[i]));
        return y;
    }

    // Wait until the lines held in lines[] (the batch's lines first..first +
    // 8 NB, of which those below nlines exist) carry tag.  Lane 7 of each
    // line holds the flag in words 2..3.  If any line is stale, the wave
    // polls the 8-byte flags alone, one line per lane, and once all match it
    // reads the lines again; a valid line cannot change before this wave
    // frees the slot.  Polling the flags rather than whole lines costs a
    // sixteenth of the traffic, and the loop's loads never land in the
    // registers that carry data, which would otherwise make the compiler
    // wait for every store of the step before the next batch's loads.
    template <int NB>
    __device__ static bool stale_lines(const u32x4 *lines, const bool *act, uint32_t p, uint64_t tag)
    {
        bool bad = false;
#pragma unroll
        for (int t = 0; t < NB; ++t)
            bad |= act[t] && p == 7 && (((uint64_t)lines[t][3] << 32) | lines[t][2]) != tag;
        return any_lane(bad);
    }
    template <int NB>
    __device__ static bool poll_flags(const RingArgs &a, Rsrc wi, uint32_t first, uint32_t nlines, uint64_t tag)
    {
        static_assert(8 * NB <= 64, "one flag per lane");
        const uint32_t lane = step_lane();
        const uint32_t fl = first + lane;
        const bool fact = lane < 8 * NB && fl < nlines;
        Watchdog wd;
        while (true) {
            __builtin_amdgcn_s_sleep(1);
            if (watchdog_expired(a, wd)) return false;
            const u32x2 f = ld64<kFifoLd>(wi, in_range(fact, fl * 128 + 120));
            if (!any_lane(fact && (((uint64_t)f[1] << 32) | f[0]) != tag)) return true;
        }
    }
    template <int NB>
    __device__ static bool await_lines(const RingArgs &a, Rsrc wi, u32x4 *lines, const uint32_t *line_of,
                                       const bool *act, uint64_t tag, uint32_t first, uint32_t nlines,
                                       bool &was_stale)
    {
        // Ordered plans take no line from a load that also brought its flag.
        was_stale = ORD || stale_lines<NB>(lines, act, step_lane() & 7u, tag);
        if (was_stale) {
            if (!poll_flags<NB>(a, wi, first, nlines, tag)) return false;
#pragma unroll
            for (int t = 0; t < NB; ++t)
                lines[t] = ld128<kFifoLd>(wi, in_range(act[t], line_of[t] * 128 + 16 * (step_lane() & 7u)));
        }
        after_observe();
        return true;
    }

    // Debug builds (AR_DEBUG_CHECK_LINES): the check words lane part p of
    // `line` carries for the message with flag `tag` (lane 7: words 0..1).
    __device__ static u32x4 check_part(uint32_t tag, uint32_t line, uint32_t p)
    {
        const uint32_t b = line * 128 + 16 * p;
        return u32x4{check_word(tag, b), check_word(tag, b + 4), check_word(tag, b + 8), check_word(tag, b + 12)};
    }
    // Check every accepted line of a batch against the writer's check words:
    // a line counts as bad if any of its eight lane parts differs.
    template <int NB>
    __device__ static void check_lines(const u32x4 *lines, const uint32_t *line_of, const bool *act, uint32_t p,
                                       uint32_t tag, bool first, DbgState *dbg)
    {
#pragma unroll
        for (int t = 0; t < NB; ++t) {
            const u32x4 w = check_part(tag, line_of[t], p);
            const bool bad = act[t] && (lines[t][0] != w[0] || lines[t][1] != w[1] ||
                                        (p < 7 && (lines[t][2] != w[2] || lines[t][3] != w[3])));
            const uint32_t n = (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(act[t] && p == 7));
            dbg->checked += n;
            dbg->first += first ? n : 0u;
            dbg->bad += groups8_set(__builtin_amdgcn_ballot_w64(bad));
        }
    }

    __device__ static bool run(const RingArgs &a, const char *src, char *dst, const char *rslot,
                               char *wslot, uint32_t len, uint64_t tag_in, uint64_t tag_out, uint32_t *lds,
                               DbgState *dbg)
    {
        const uint32_t lane = step_lane();
        const uint32_t p = lane & 7u, ls = lane >> 3;
        const bool chk = DBG && dbg->check;
        const Rsrc rin = make_rsrc(src, (uint64_t)len * E);
        const Rsrc rout = make_rsrc(dst, (uint64_t)len * E);
        // rslot: the incoming FIFO slot, or for a peer read the chain
        // start's input at this message's elements (then `wire` holds it in
        // the data type)
        const Rsrc wi = make_rsrc(rslot, kRecvPeer ? (uint64_t)len * E : a.slot_bytes);
        const Rsrc wo = make_rsrc(wslot, a.slot_bytes);
        if constexpr (!kRelayout) {
            // One line format in and out: the lane part maps to the same elements.
            constexpr uint32_t epl = (kRecvRS || kSendRS) ? kEplRS : kEplAG;
            constexpr uint32_t epart = 16 / ((kRecvRS || kSendRS) ? 4 : E);  // elements per full part
            const uint32_t nlines = (len + epl - 1) / epl;
            const uint32_t full = p < 7 ? epart : epart / 2;
            // Unit t of the batch at line `base`: the lane's line, and how
            // many of its lane part's elements exist.
            auto unit = [&](uint32_t base, int t, uint32_t &line, bool &act, uint32_t &nval) {
                line = base + 8 * t + ls;
                act = line < nlines;
                const uint32_t e0 = line * epl + p * epart;
                nval = act && e0 < len ? (len - e0 < full ? len - e0 : full) : 0;
            };
            auto issue = [&](uint32_t base, u32x4 *in, u32x4 *wire) {
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    uint32_t line, nval;
                    bool act;
                    unit(base, t, line, act, nval);
                    if (kLoadIn) in[t] = load_whole<epart>(rin, (line * epl + p * epart) * E, p, nval, full);
                    if (kRecvRS || kRecvAG) wire[t] = ld128<kFifoLd>(wi, in_range(act, line * 128 + 16 * p));
                    if (kRecvPeer) wire[t] = load_whole<epart>(wi, (line * epl + p * epart) * E, p, nval, full);
                }
            };
            // Lines are written in groups of kGroup batches; one drain per
            // group makes the group's data complete before its flags go out.
            for (uint32_t gbase = 0; gbase < nlines; gbase += 8 * U * kGroup) {
                const uint32_t gend = gbase + 8 * U * kGroup < nlines ? gbase + 8 * U * kGroup : nlines;
                u32x4 in[U], wire[U];
#pragma unroll
                for (int t = 0; t < U; ++t) in[t] = wire[t] = u32x4{0, 0, 0, 0};
                issue(gbase, in, wire);
                for (uint32_t base = gbase; base < gend; base += 8 * U) {
                    uint32_t line_of[U], nval[U];
                    bool act[U];
#pragma unroll
                    for (int t = 0; t < U; ++t) unit(base, t, line_of[t], act[t], nval[t]);
                    if (kRecvRS || kRecvAG) {
                        bool stale = false;
                        if (!await_lines<U>(a, wi, wire, line_of, act, tag_in, base, nlines, stale)) return false;
                        if constexpr (DBG) {
                            if (dbg->trace && dbg->tr.t_recv == 0) {
                                dbg->tr.t_recv = now_ticks();
                                dbg->tr.polls = stale ? 1u : 0u;
                            }
                            if (chk) check_lines<U>(wire, line_of, act, p, (uint32_t)tag_in, !stale, dbg);
                        }
                    }
                    // All inputs in place before the first store: a cut-part
                    // load between stores would make the stores wait.
                    if (kLoadIn) {
#pragma unroll
                        for (int t = 0; t < U; ++t)
                            in[t] = part_value<epart>(rin, (line_of[t] * epl + p * epart) * E, p, nval[t], full, in[t]);
                    }
                    if (kRecvPeer) {
#pragma unroll
                        for (int t = 0; t < U; ++t)
                            wire[t] = part_value<epart>(wi, (line_of[t] * epl + p * epart) * E, p, nval[t], full,
                                                        wire[t]);
                    }
                    // The next batch's loads go out before this batch's
                    // stores: the vector memory counter retires in issue
                    // order, so a load issued after a store cannot be waited
                    // for without waiting for the store as well.
                    u32x4 nin[U], nwire[U];
#pragma unroll
                    for (int t = 0; t < U; ++t) nin[t] = nwire[t] = u32x4{0, 0, 0, 0};
                    if (base + 8 * U < gend) issue(base + 8 * U, nin, nwire);
#pragma unroll
                    for (int t = 0; t < U; ++t) {
                        const uint32_t e0 = line_of[t] * epl + p * epart;
                        u32x4 out;
                        if (kRecvPeer && E == 2 && !kSendRS) out = peer_y8(wire[t], in[t]);
                        else if (kSendRS || kReduceToY) out = rs_reduce(wire[t], in[t]);
                        else if (kCopyInToY) out = in[t];
                        else out = wire[t];
                        if (kWriteOut) {
                            if (KIND == kRecvReduceCopy && E == 2) {
                                // bf16 owner: round the fp32 sums once, 4 values per lane part
                                const u32x4 y = {pack_bf16(as_f32(out[0]), as_f32(out[1])),
                                                 pack_bf16(as_f32(out[2]), as_f32(out[3])), 0, 0};
                                store_part<epart>(rout, e0 * E, y, p, nval[t], full);
                            } else {
                                store_part<epart>(rout, e0 * E, out, p, nval[t], full);
                            }
                        }
                        if (kSendRS || kSendAG) put_data(wo, line_of[t], p, act[t], chk ? check_part((uint32_t)tag_out, line_of[t], p) : out);
                    }
#pragma unroll
                    for (int t = 0; t < U; ++t) {
                        in[t] = nin[t];
                        wire[t] = nwire[t];
                    }
                }
                if (kSendRS || kSendAG) {
                    if constexpr (DBG)
                        if (dbg->trace && dbg->tr.t_issued == 0) dbg->tr.t_issued = now_ticks();
                    drain_vmem();
                    if constexpr (DBG)
                        if (dbg->trace && dbg->tr.t_drained == 0) dbg->tr.t_drained = now_ticks();
                    put_flags(wo, gbase, gend, lane, tag_out);
                    if constexpr (DBG)
                        if (dbg->trace && dbg->tr.t_posted == 0) dbg->tr.t_posted = now_ticks();
                }
            }
            return true;
        } else {
            // bf16 recvReduceCopySend: 16 reduce-scatter lines (480 elements, two
            // wave loads) become 8 all-gather lines (one wave store) per round.
            const uint32_t nlines_ag = (len + kEplAG - 1) / kEplAG;
            for (uint32_t gbase = 0; gbase < nlines_ag; gbase += 8 * kGroup) {
                for (uint32_t agb = gbase; agb < gbase + 8 * kGroup && agb < nlines_ag; agb += 8) {
                    // Phase 1: receive 16 RS lines, reduce, stage bf16 results in LDS.
                    u32x4 in[2], wire[2];
                    uint32_t line_of[2], nval[2];
                    bool act[2];
                    const uint32_t rs_nlines = (len + kEplRS - 1) / kEplRS;
                    const uint32_t full = p < 7 ? 4u : 2u;
    #pragma unroll
                    for (int t = 0; t < 2; ++t) {
                        line_of[t] = 2 * agb + 8 * t + ls;
                        act[t] = line_of[t] < rs_nlines;
                        const uint32_t e0 = line_of[t] * kEplRS + p * 4;
                        nval[t] = act[t] && e0 < len ? (len - e0 < full ? len - e0 : full) : 0;
                        in[t] = load_whole<4>(rin, e0 * E, p, nval[t], full);
                        wire[t] = ld128<kFifoLd>(wi, in_range(act[t], line_of[t] * 128 + 16 * p));
                    }
                    bool stale = false;
                    if (!await_lines<2>(a, wi, wire, line_of, act, tag_in, 2 * agb, rs_nlines, stale)) return false;
                    if constexpr (DBG) {
                        if (dbg->trace && dbg->tr.t_recv == 0) {
                            dbg->tr.t_recv = now_ticks();
                            dbg->tr.polls = stale ? 1u : 0u;
                        }
                        if (chk) check_lines<2>(wire, line_of, act, p, (uint32_t)tag_in, !stale, dbg);
                    }
    #pragma unroll
                    for (int t = 0; t < 2; ++t) {
                        // Element index of this lane's first value within the 480-block.
                        const uint32_t loc = (8 * t + ls) * kEplRS + p * 4;
                        const uint32_t e0 = line_of[t] * kEplRS + p * 4;
                        u32x4 acc = rs_reduce(wire[t], part_value<4>(rin, e0 * E, p, nval[t], full, in[t]));
                        lds[loc / 2] = pack_bf16(as_f32(acc[0]), as_f32(acc[1]));
                        if (p < 7) lds[loc / 2 + 1] = pack_bf16(as_f32(acc[2]), as_f32(acc[3]));
                    }
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
                    // Phase 2: read back in the 60-per-line layout, write output and AG line.
                    const uint32_t line = agb + ls;
                    const bool act2 = line < nlines_ag;
                    const uint32_t full2 = p < 7 ? 8u : 4u;
                    const uint32_t e0 = line * kEplAG + p * 8;
                    const uint32_t n2 = act2 && e0 < len ? (len - e0 < full2 ? len - e0 : full2) : 0;
                    const uint32_t loc = ls * kEplAG + p * 8;
                    u32x4 y = {lds[loc / 2], lds[loc / 2 + 1], 0, 0};
                    if (p < 7) {
                        y[2] = lds[loc / 2 + 2];
                        y[3] = lds[loc / 2 + 3];
                    }
                    store_part<8>(rout, e0 * E, y, p, n2, full2);
                    put_data(wo, line, p, act2, chk ? check_part((uint32_t)tag_out, line, p) : y);
                    // LDS is rewritten by the next round only after every lane has read it.
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
                }
                if constexpr (DBG)
                    if (dbg->trace && dbg->tr.t_issued == 0) dbg->tr.t_issued = now_ticks();
                drain_vmem();
                if constexpr (DBG)
                    if (dbg->trace && dbg->tr.t_drained == 0) dbg->tr.t_drained = now_ticks();
                const uint32_t gend = gbase + 8 * kGroup < nlines_ag ? gbase + 8 * kGroup : nlines_ag;
                put_flags(wo, gbase, gend, lane, tag_out);
                if constexpr (DBG)
                    if (dbg->trace && dbg->tr.t_posted == 0) dbg->tr.t_posted = now_ticks();
            }
            return true;
        }
    }
};

constexpr uint32_t kLdsWordsPerWave = 240;  // 480 bf16 values

template <int DT, int KIND, bool DBG, int LU, bool ORD>
__device__ __forceinline__ bool ll128_step(Ring &g, const char *src, char *dst, const char *peer_src, uint32_t len,
                                           uint32_t *lds)
{
    const RingArgs &a = *g.a;
    constexpr bool recv = KindTraits<KIND>::kRecvRS || KindTraits<KIND>::kRecvAG;
    constexpr bool send = KindTraits<KIND>::kSendRS || KindTraits<KIND>::kSendAG;
    const char *rslot = nullptr;
    char *wslot = nullptr;
    // LL128 runs out of vector registers first, so it derives the slot from
    // the message index instead of carrying the slot counters.
    if (recv) rslot = slot_ptr(const_cast<char *>(g.fifo_in), (uint32_t)(g.m_in % a.depth), a);
    if (KindTraits<KIND>::kRecvPeer) rslot = peer_src;
    if (send) {
        if (!acquire_send_slot(g)) return false;
        wslot = slot_ptr(g.fifo_out, (uint32_t)(g.m_out % a.depth), a);
    }
    if constexpr (DBG)
        if (send) debug_jitter(a, g.m_out ^ ((uint64_t)g.r << 40) ^ ((uint64_t)g.c << 48));
    const bool skip = DBG && send && skip_this_post(g);
    // A skipped post: write the data but a flag from the previous message.
    const uint64_t tag_out = skip ? g.m_out : g.m_out + 1;
    if (!LL128Step<DT, KIND, DBG, LU, ORD>::run(a, src, dst, rslot, wslot, len, g.m_in + 1, tag_out, lds, &g.dbg))
        return false;
    if (send) advance_out(g);
    if (recv) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        flag_store(g.head_in, g.m_in + 1);
        advance_in(g);
    }
    return true;
}

// ===================================================================== kernel

// Debug builds: store the step's trace record, one field per store from
// lane 0 (records beyond the rank's share of the buffer are dropped).  A
// field picked by lane index would read the record as an array with a
// variable index, which puts it, and everything it lives in, into scratch.
__device__ __forceinline__ void write_trace(const Ring &g)
{
    const RingArgs &a = *g.a;
    const bool keep = lane_id() == 0 && g.dbg.step < a.trace_per_rank;
    const uint64_t rec = (uint64_t)g.r * a.trace_per_rank + g.dbg.step;
    const Rsrc rt = make_rsrc(a.trace + rec * kTraceFields, kTraceFields * 8);
    const StepTrace &t = g.dbg.tr;
    auto put = [&](uint32_t i, uint64_t v) {
        st64<kPolPlain>(rt, in_range(keep, i * 8), u32x2{(uint32_t)v, (uint32_t)(v >> 32)});
    };
    put(0, t.t_begin);
    put(1, t.t_recv);
    put(2, t.polls);
    put(3, t.t_issued);
    put(4, t.t_drained);
    put(5, t.t_posted);
    put(6, t.msg);
    put(7, t.kind);
}

template <int PROTO, int DT, bool DAG, bool DBG, int LU, bool ORD, int KIND>
__device__ __forceinline__ bool do_step(Ring &g, const char *src, char *dst, char *peer_dst, const char *peer_src,
                                        uint32_t len, uint32_t *lds)
{
    if constexpr (DBG) {
        if (g.dbg.trace) {
            g.dbg.tr = StepTrace{};
            g.dbg.tr.t_begin = now_ticks();
            g.dbg.tr.kind = KIND;
            constexpr bool send = KindTraits<KIND>::kSendRS || KindTraits<KIND>::kSendAG;
            g.dbg.tr.msg = send ? g.m_out : g.m_in;
        }
    }
    bool ok;
    if (PROTO == AR_PROTO_SIMPLE) ok = simple_step<DT, KIND, DAG, DBG>(g, src, dst, peer_dst, peer_src, len);
    else if (PROTO == AR_PROTO_LL) ok = ll_step<DT, KIND, DBG>(g, src, dst, peer_src, len);
    else ok = ll128_step<DT, KIND, DBG, LU, ORD>(g, src, dst, peer_src, len, lds);
    if constexpr (DBG) {
        if (g.dbg.trace) {
            write_trace(g);
            ++g.dbg.step;
        }
    }
    return ok;
}

// All steps of one run for one wave; false if the wave had to give up.
template <int PROTO, int DT, bool DAG, bool DBG, int LU, bool ORD>
__device__ __forceinline__ bool ring_steps(Ring &g, uint32_t *lds)
{
    constexpr uint32_t E = Elem<DT>::E;
    const RingArgs &a = *g.a;
    const uint32_t N = g.N, r = g.r, c = g.c, w = g.w;

    // Step schedule per collective (segment handled at ring step k):
    //   AllReduce      k = 0 .. 2N-2, segment (r - k) mod N, owner of s is s-1
    //   ReduceScatter  k = 0 .. N-1,  segment (r - 1 - k) mod N, owner of s is s
    //   AllGather      k = 0 .. N-1,  segment (r - k) mod N, starting from the own block
    // In the peer-direct mode (DAG) a reduction chain has no step 0: at step
    // 1 the second rank reads the chain start's input from that rank's buffer.
    const char *src = a.src[r];
    char *dst = a.dst[r];
    char *peer = DAG ? a.dst[r + 1 == N ? 0 : r + 1] : nullptr;             // the next rank's output
    const char *prev_src = DAG ? a.src[r == 0 ? N - 1 : r - 1] : nullptr;  // the previous rank's input
    const uint32_t coll = a.coll;
    const bool peer_start = DAG && coll != AR_COLL_ALLGATHER;
    const uint32_t nsteps = coll == AR_COLL_ALLREDUCE ? 2 * N - 1 : N;
    const uint32_t k0 = peer_start ? 1u : 0u;
    uint32_t s0 = coll == AR_COLL_REDUCESCATTER ? (r + N - 1) % N : r;
    if (peer_start) s0 = s0 == 0 ? N - 1 : s0 - 1;
    // A wave's elements of chunk j sit at the same offset (rel) inside every
    // segment; only the segment base and, for the one partial segment and
    // the empty ones after it, the length change from step to step.  So the
    // clamps are done once per chunk and a step costs a few scalar ops.
    const uint64_t last_lo = (uint64_t)(N - 1) * a.seg;
    const uint64_t c_lo = (uint64_t)c * a.cs;
    for (uint32_t j = 0; j < a.nchunks; ++j) {
        const uint64_t ck_lo = c_lo + (uint64_t)j * a.chunk;
        const uint64_t rel = ck_lo + (uint64_t)w * a.kw;
        uint64_t hi = c_lo + a.cs;
        if (ck_lo + a.chunk < hi) hi = ck_lo + a.chunk;
        if (rel + a.kw < hi) hi = rel + a.kw;
        const uint64_t hi_full = hi < a.seg ? hi : a.seg;
        const uint64_t hi_part = hi < a.part ? hi : a.part;
        const uint32_t len_full = hi_full > rel ? (uint32_t)(hi_full - rel) : 0u;
        const uint32_t len_part = hi_part > rel ? (uint32_t)(hi_part - rel) : 0u;
        uint32_t s = s0;
        uint64_t seg_lo = (uint64_t)s0 * a.seg;
        for (uint32_t k = k0; k < nsteps; ++k) {
            const uint32_t len = s < a.full_segs ? len_full : (s == a.full_segs ? len_part : 0u);
            const uint64_t lo = seg_lo + rel;
            // ReduceScatter writes, and AllGather reads, one block-sized buffer.
            const uint64_t in_e = len ? (coll == AR_COLL_ALLGATHER ? rel : lo) : 0;
            const uint64_t out_e = len ? (coll == AR_COLL_REDUCESCATTER ? rel : lo) : 0;
            if (s == 0) {
                s = N - 1;
                seg_lo = last_lo;
            } else {
                --s;
                seg_lo -= a.seg;
            }
            const char *s_ptr = src + in_e * E;
            char *d_ptr = dst + out_e * E;
            char *p_ptr = DAG ? peer + out_e * E : nullptr;
            const char *q_ptr = DAG ? prev_src + in_e * E : nullptr;
            bool ok;
            if constexpr (DAG) {
                if (peer_start && k == 1) {
                    if (coll == AR_COLL_ALLREDUCE && N == 2)
                        ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kPeerReduceCopySend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                    else if (N == 2)
                        ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kPeerReduceCopy>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                    else
                        ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kPeerReduceSend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                    if (!ok) return false;
                    continue;
                }
            }
            if (coll == AR_COLL_ALLREDUCE) {
                if (k == 0) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kSend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else if (k < N - 1) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvReduceSend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else if (k == N - 1) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvReduceCopySend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else if (k < 2 * N - 2) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvCopySend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvCopy>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
            } else if (coll == AR_COLL_REDUCESCATTER) {
                if (k == 0) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kSend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else if (k < N - 1) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvReduceSend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvReduceCopy>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
            } else {
                if (k == 0) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kCopySend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else if (k < N - 1) ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvCopySend>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
                else ok = do_step<PROTO, DT, DAG, DBG, LU, ORD, kRecvCopy>(g, s_ptr, d_ptr, p_ptr, q_ptr, len, lds);
            }
            if (!ok) return false;
        }
    }
    return true;
}

// DBG: the debug hooks (AR_DEBUG_*) are compiled in; a plan without debug
// flags runs the kernel without them, whose steps carry no test-only code.
// LU: the LL128 batch width (LL128Step); 2 for the other protocols.
// ORD: LL128 reads a batch only after its flags (AR_PLAN_LL128_ORDERED); a
// build of its own, since even an untaken test of a run-time flag costs the
// two-access step 0.26 us per hop.
template <int PROTO, int DT, bool DAG, bool DBG, int LU, bool ORD>
__global__ __launch_bounds__(1024) void ring_kernel(RingArgs a)
{
    __shared__ uint32_t lds_all[(PROTO == AR_PROTO_LL128 && DT == AR_BFLOAT16) ? AR_MAX_WAVES * kLdsWordsPerWave : 1];
    const uint32_t N = a.nranks, C = a.nchannels, W = a.nwaves;
    const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t b = blockIdx.x;
    uint32_t c, r;
    if (a.placement == AR_PLACE_CHANNEL_LOCAL) {
        r = b / C;
        c = b % C;
    } else {
        c = b / N;
        r = b % N;
    }
    const uint32_t rprev = (r + N - 1) % N;
    const uint64_t conn_out = ((uint64_t)c * W + w) * N + r;
    const uint64_t conn_in = ((uint64_t)c * W + w) * N + rprev;

    Ring g;
    g.a = &a;
    g.N = N;
    g.r = r;
    g.c = c;
    g.w = w;
    g.tail_out = a.flags + conn_out * kConnFlagU64;
    g.head_out = g.tail_out + kFlagLineU64;
    g.tail_in = a.flags + conn_in * kConnFlagU64;
    g.head_in = g.tail_in + kFlagLineU64;
    g.fifo_out = a.fifo + conn_out * a.depth * a.slot_bytes;
    g.fifo_in = a.fifo + conn_in * a.depth * a.slot_bytes;
    // Each wave keeps its message epoch in device memory, so a launch
    // captured in a graph and replayed continues the counters where the last
    // run left them.  It is read here together with the head counter of the
    // outgoing link (whose final value from the previous run frees the first
    // slots), so both cost one round trip.  Only this wave reads or writes
    // its epoch, and every member of a ring sends and receives the same
    // number of messages per run, so the members' epochs stay equal without
    // any exchange; the next run's value is stored at once, which keeps
    // nothing alive across the loop.  (A wave that gives up leaves the plan
    // in its timeout state, which only ar_plan_reset clears, zeroing every
    // epoch.)
    uint64_t *epoch_p = g.tail_out + kEpochU64;
    // The abort word goes out with them: a wave that tested it only after
    // the first two had arrived would start every run one round trip later.
    const uint64_t epoch_word = flag_load(epoch_p);
    const uint64_t head_word = flag_load(g.head_out);
    const uint32_t abort_word = __hip_atomic_load(a.ctl + kCtlAbort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t epoch = uniform64(epoch_word);
    g.head_seen = uniform64(head_word);
    const bool aborted = __builtin_amdgcn_readfirstlane(abort_word) != 0;
    after_observe();
    {
        // messages per chunk: 2N-2 (AllReduce) or N-1, one fewer when a
        // reduction chain starts with a peer read (stored by every lane)
        const uint64_t per_chunk = (a.coll == AR_COLL_ALLREDUCE ? 2 * N - 2 : N - 1) -
                                   (DAG && a.coll != AR_COLL_ALLGATHER ? 1 : 0);
        flag_store(epoch_p, epoch + (uint64_t)a.nchunks * per_chunk);
    }
    g.m_out = epoch;
    g.m_in = epoch;
    g.slot_out = g.slot_in = (uint32_t)(epoch % a.depth);
    g.tail_seen = 0;
    uint32_t *lds = lds_all + ((PROTO == AR_PROTO_LL128 && DT == AR_BFLOAT16) ? w * kLdsWordsPerWave : 0);

    g.dbg = DbgState{};
    if constexpr (DBG) {
        g.dbg.check = (a.debug & AR_DEBUG_CHECK_LINES) != 0 && PROTO != AR_PROTO_SIMPLE;
        g.dbg.trace = (a.debug & AR_DEBUG_TRACE) != 0 && a.trace != nullptr && c == 0 && w == 0;
    }

    // A previous run that timed out leaves the abort word raised: do nothing.
    if (aborted) return;
    ring_steps<PROTO, DT, DAG, DBG, LU, ORD>(g, lds);
    if constexpr (DBG) {
        // One lane adds the wave's line-check counts (nothing follows).
        if (g.dbg.check && lane_id() == 0) {
            uint64_t *cnt = (uint64_t *)(a.ctl + kCtlLinesChecked);
            __hip_atomic_fetch_add(cnt, (uint64_t)g.dbg.checked, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            cnt = (uint64_t *)(a.ctl + kCtlLinesFirst);
            __hip_atomic_fetch_add(cnt, (uint64_t)g.dbg.first, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            cnt = (uint64_t *)(a.ctl + kCtlLinesBad);
            __hip_atomic_fetch_add(cnt, (uint64_t)g.dbg.bad, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// ===================================================================== direct
//
// Two-shot direct AllReduce: workgroup b works on segment s = b mod N (part
// b / N of its parts); a thread loads one 16-byte unit of segment s from
// every rank (ranks s, s+1, ..., s+N-1 in that order), sums them in that
// chain order -- the same additions, in the same order, as the ring's
// reduce-scatter -- and stores the result to every rank.  Every element is
// read once per rank and written once per rank: the compulsory 2 N S bytes,
// no FIFOs, no flags, no waits.  In place is safe: each element is read and
// then written by the same thread.
//
// The same kernel runs the other collectives directly: ReduceScatter sums
// block s along the chain that starts at rank s+1 (the ring's order for a
// block that ends at rank s) and writes it to rank s only; AllGather copies
// rank s's block to block s of every rank.

template <int DT, int NMAX, int U>
__global__ __launch_bounds__(1024) void direct_kernel(RingArgs a)
{
    constexpr uint32_t E = Elem<DT>::E;
    constexpr uint32_t A = Elem<DT>::A;
    const uint32_t N = a.nranks;
    const uint32_t parts = a.nchannels;
    const uint32_t s = blockIdx.x % N;
    const uint32_t part = blockIdx.x / N;
    const uint32_t coll = a.coll;
    const uint32_t nsrc = coll == AR_COLL_ALLGATHER ? 1u : N;       // chain length
    const uint32_t first = coll == AR_COLL_REDUCESCATTER ? s + 1 : s;  // chain start rank
    const uint32_t nout = coll == AR_COLL_REDUCESCATTER ? 1u : N;    // ranks written
    const uint64_t seg_lo = (uint64_t)s * a.seg;
    if (seg_lo >= a.count) return;
    const uint64_t seg_hi = seg_lo + a.seg < a.count ? seg_lo + a.seg : a.count;
    const uint64_t len = seg_hi - seg_lo;
    const uint64_t nfull_all = len / A;
    const uint32_t rem = (uint32_t)(len % A);
    const uint32_t tid = threadIdx.x, nth = blockDim.x;

    // Rank j of the chain is rank (first + j) mod N.  AllGather reads a
    // block-sized source, ReduceScatter writes a block-sized destination.
    // A descriptor covers `bytes` from byte `off` of the segment: buffer
    // offsets are 32-bit, so a segment is walked in windows of kWinUnits
    // units (one window up to 1 GiB per segment).
    auto in_rsrc = [&](uint32_t j, uint64_t off, uint64_t bytes) {
        const uint32_t r = (first + j) % N;
        return make_rsrc(a.src[r] + (coll == AR_COLL_ALLGATHER ? 0 : seg_lo * E) + off, bytes);
    };
    auto out_rsrc = [&](uint32_t i, uint64_t off, uint64_t bytes) {
        const uint32_t r = coll == AR_COLL_REDUCESCATTER ? s : i;
        return make_rsrc(a.dst[r] + (coll == AR_COLL_REDUCESCATTER ? 0 : seg_lo * E) + off, bytes);
    };
    constexpr uint64_t kWinUnits = 1ull << 26;

    auto chain = [&](const u32x4 *v, float *acc) {
        if (E == 4) {
            for (int i = 0; i < 4; ++i) acc[i] = as_f32(v[0][i]);
        } else {
            for (int i = 0; i < 4; ++i) {
                acc[2 * i] = bf16_lo(v[0][i]);
                acc[2 * i + 1] = bf16_hi(v[0][i]);
            }
        }
#pragma unroll
        for (int j = 1; j < NMAX; ++j) {
            if ((uint32_t)j < nsrc) {
                if (E == 4) {
                    for (int i = 0; i < 4; ++i) acc[i] = acc[i] + as_f32(v[j][i]);
                } else {
                    for (int i = 0; i < 4; ++i) {
                        acc[2 * i] = acc[2 * i] + bf16_lo(v[j][i]);
                        acc[2 * i + 1] = acc[2 * i + 1] + bf16_hi(v[j][i]);
                    }
                }
            }
        }
    };
    auto narrow = [&](const float *acc) {
        u32x4 y;
        if (E == 4) {
            for (int i = 0; i < 4; ++i) y[i] = as_u32(acc[i]);
        } else {
            for (int i = 0; i < 4; ++i) y[i] = pack_bf16(acc[2 * i], acc[2 * i + 1]);
        }
        return y;
    };

    for (uint64_t w0 = 0; w0 < nfull_all; w0 += kWinUnits) {
        const uint32_t nfull = (uint32_t)(nfull_all - w0 < kWinUnits ? nfull_all - w0 : kWinUnits);
        const uint64_t woff = w0 * 16, wbytes = (uint64_t)nfull * 16;
        for (uint32_t base = part * nth * U; base < nfull; base += parts * nth * U) {
            u32x4 v[U][NMAX];
#pragma unroll
            for (int j = 0; j < NMAX; ++j) {
                if ((uint32_t)j < nsrc) {
                    const Rsrc rin = in_rsrc(j, woff, wbytes);
#pragma unroll
                    for (int t = 0; t < U; ++t) {
                        const uint32_t u = base + t * nth + tid;
                        v[t][j] = ld128<kInPol>(rin, in_range(u < nfull, u * 16));
                    }
                }
            }
            u32x4 y[U];
#pragma unroll
            for (int t = 0; t < U; ++t) {
                if (coll == AR_COLL_ALLGATHER) {
                    y[t] = v[t][0];  // a copy keeps every bit, NaN payloads included
                } else {
                    float acc[A];
                    chain(v[t], acc);
                    y[t] = narrow(acc);
                }
            }
#pragma unroll
            for (int r = 0; r < NMAX; ++r) {
                if ((uint32_t)r < nout) {
                    const Rsrc rout = out_rsrc(r, woff, wbytes);
#pragma unroll
                    for (int t = 0; t < U; ++t) {
                        const uint32_t u = base + t * nth + tid;
                        st128<kOutPol>(rout, in_range(u < nfull, u * 16), y[t]);
                    }
                }
            }
        }
    }
    if (rem && part == 0 && tid == 0) {
        // Partial last unit of the buffer: element-wise loads and stores
        // (every index below is a compile-time constant after unrolling).
        u32x4 v[NMAX];
#pragma unroll
        for (int j = 0; j < NMAX; ++j) {
            u32x4 x = {0, 0, 0, 0};
            if ((uint32_t)j < nsrc) {
                const Rsrc rin = in_rsrc(j, nfull_all * 16, (uint64_t)rem * E);
#pragma unroll
                for (int i = 0; i < (int)A; ++i) {
                    if ((uint32_t)i < rem) {
                        if (E == 4) x[i] = ld32<kInPol>(rin, 4 * i);
                        else x[i >> 1] |= ld16<kInPol>(rin, 2 * i) << ((i & 1) * 16);
                    }
                }
            }
            v[j] = x;
        }
        u32x4 y = v[0];
        if (coll != AR_COLL_ALLGATHER) {
            float acc[A];
            chain(v, acc);
            y = narrow(acc);
        }
#pragma unroll
        for (int r = 0; r < NMAX; ++r) {
            if ((uint32_t)r < nout) {
                const Rsrc rout = out_rsrc(r, nfull_all * 16, (uint64_t)rem * E);
#pragma unroll
                for (int i = 0; i < (int)A; ++i) {
                    if ((uint32_t)i < rem) {
                        if (E == 4) st32<kOutPol>(rout, 4 * i, y[i]);
                        else st16<kOutPol>(rout, 2 * i, (y[i >> 1] >> ((i & 1) * 16)) & 0xFFFFu);
                    }
                }
            }
        }
    }
}

// ------------------------------------------------------------------ helpers

__global__ void fill_u32_kernel(uint32_t *p, size_t n, uint32_t v)
{
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// Streaming copy of nunits 16-byte units (both ends 16-byte aligned), four
// units per thread and iteration with every load of an iteration issued
// before its stores, walked in 1 GiB windows so buffer offsets stay 32-bit;
// then `tail` (< 16) trailing bytes.  On MI355X this shape moves 1 GiB to
// 1 GiB at about 6.1 TB/s of reads plus writes.
__global__ __launch_bounds__(256) void copy_kernel(const char *src, char *dst, uint64_t nunits, uint32_t tail)
{
    constexpr int U = 4;
    constexpr uint64_t kWin = 1ull << 26;
    const uint32_t nth = blockDim.x * gridDim.x;
    for (uint64_t w0 = 0; w0 < nunits; w0 += kWin) {
        const uint32_t n = (uint32_t)(nunits - w0 < kWin ? nunits - w0 : kWin);
        const Rsrc rs = make_rsrc(src + w0 * 16, (uint64_t)n * 16);
        const Rsrc rd = make_rsrc(dst + w0 * 16, (uint64_t)n * 16);
        for (uint32_t base = blockIdx.x * blockDim.x * U; base < n; base += nth * U) {
            u32x4 v[U];
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const uint32_t u = base + t * blockDim.x + threadIdx.x;
                v[t] = ld128<kPolNt>(rs, in_range(u < n, u * 16));
            }
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const uint32_t u = base + t * blockDim.x + threadIdx.x;
                st128<kPolNt>(rd, in_range(u < n, u * 16), v[t]);
            }
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < tail) dst[nunits * 16 + threadIdx.x] = src[nunits * 16 + threadIdx.x];
}

__global__ void bf16_round_kernel(const float *in, uint16_t *out, size_t n)
{
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        out[i] = (uint16_t)bf16_rne(in[i]);
}

typedef void (*RingFn)(RingArgs);

// dag: the peer-direct mode (chains start with a peer read; the Simple
// ring also writes its all-gather into the next rank's output).
template <int DT, bool DBG, bool ORD, bool DAG>
__host__ RingFn ll128_fn(bool wide)
{
    return wide ? ring_kernel<AR_PROTO_LL128, DT, DAG, DBG, 4, ORD> : ring_kernel<AR_PROTO_LL128, DT, DAG, DBG, 2, ORD>;
}

template <int DT, bool DBG>
__host__ RingFn ring_fn_of(int proto, bool dag, bool wide, bool ordered)
{
    if (proto == AR_PROTO_LL)
        return dag ? ring_kernel<AR_PROTO_LL, DT, true, DBG, 2, false> : ring_kernel<AR_PROTO_LL, DT, false, DBG, 2, false>;
    if (proto == AR_PROTO_LL128) {
        if (dag) return ordered ? ll128_fn<DT, DBG, true, true>(wide) : ll128_fn<DT, DBG, false, true>(wide);
        return ordered ? ll128_fn<DT, DBG, true, false>(wide) : ll128_fn<DT, DBG, false, false>(wide);
    }
    return dag ? ring_kernel<AR_PROTO_SIMPLE, DT, true, DBG, 2, false> : ring_kernel<AR_PROTO_SIMPLE, DT, false, DBG, 2, false>;
}

// dbg: a plan with debug flags runs the instance with the debug hooks.
// wide: LL128 with four-access batches; ordered: AR_PLAN_LL128_ORDERED.
__host__ RingFn ring_fn(int proto, int dtype, bool dag, bool dbg, bool wide, bool ordered)
{
    if (dtype == AR_FLOAT32)
        return dbg ? ring_fn_of<AR_FLOAT32, true>(proto, dag, wide, ordered)
                   : ring_fn_of<AR_FLOAT32, false>(proto, dag, wide, ordered);
    return dbg ? ring_fn_of<AR_BFLOAT16, true>(proto, dag, wide, ordered)
               : ring_fn_of<AR_BFLOAT16, false>(proto, dag, wide, ordered);
}

// LL128 takes four-access batches when one wave's message spans more than
// one two-access batch (16 lines of 30 fp32 reduce-scatter partials).
__host__ bool ll128_wide(const ar_plan_info &info)
{
    return info.proto == AR_PROTO_LL128 && (info.wave_elems * 4 + 119) / 120 > 16;
}

// unroll: 16-byte units per thread and iteration.  Two keep more loads in
// flight, which pays while the data is cache-resident; one streams faster
// from HBM, where the fastest grid is also small (about 800-1000 waves at
// 128 MiB x 8 ranks) and keeps fewer DRAM streams open.
__host__ RingFn direct_fn(int dtype, int nranks, int unroll)
{
    if (dtype == AR_FLOAT32) {
        if (nranks > 8) return direct_kernel<AR_FLOAT32, 16, 1>;
        return unroll == 2 ? direct_kernel<AR_FLOAT32, 8, 2> : direct_kernel<AR_FLOAT32, 8, 1>;
    }
    if (nranks > 8) return direct_kernel<AR_BFLOAT16, 16, 1>;
    return unroll == 2 ? direct_kernel<AR_BFLOAT16, 8, 2> : direct_kernel<AR_BFLOAT16, 8, 1>;
}

}  // namespace dev

int launch_ring(const ar_plan_info &info, const RingArgs &args, void *stream)
{
    dev::RingFn fn = info.algo == AR_ALGO_DIRECT ? dev::direct_fn(info.dtype, info.nranks, info.direct_unroll)
                                                 : dev::ring_fn(info.proto, info.dtype, info.peer_direct != 0,
                                                                args.debug != 0, dev::ll128_wide(info),
                                                                args.ll128_ordered != 0);
    RingArgs a = args;
    void *kargs[] = {&a};
    hipError_t e = hipLaunchKernel((const void *)fn, dim3((unsigned)info.grid), dim3((unsigned)info.block), kargs,
                                   0, (hipStream_t)stream);
    return e == hipSuccess ? AR_OK : AR_ERR_HIP;
}

// The smallest co-residency of the protocol's kernel variants.
int ring_occupancy(int proto, int dtype, int block, int *blocks_per_cu)
{
    int best = 1 << 30;
    for (int v = 0; v < 16; ++v) {
        dev::RingFn fn = dev::ring_fn(proto, dtype, (v & 1) != 0, (v & 2) != 0, (v & 4) != 0, (v & 8) != 0);
        int n = 0;
        hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, (const void *)fn, block, 0);
        if (e != hipSuccess) return AR_ERR_HIP;
        if (n < best) best = n;
    }
    *blocks_per_cu = best;
    return AR_OK;
}

int launch_fill_u32(uint32_t *p, size_t n, uint32_t value, void *stream)
{
    if (n == 0) return AR_OK;
    size_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    void *kargs[] = {&p, &n, &value};
    return hipLaunchKernel((const void *)dev::fill_u32_kernel, dim3((unsigned)blocks), dim3(256), kargs, 0,
                           (hipStream_t)stream) == hipSuccess ? AR_OK : AR_ERR_HIP;
}

int launch_copy(const void *src, void *dst, size_t bytes, void *stream)
{
    if (bytes == 0 || src == dst) return AR_OK;
    // Both ends are 16-byte aligned (every rank buffer is checked for it).
    const uint64_t nunits = bytes / 16;
    const uint32_t tail = (uint32_t)(bytes % 16);
    uint64_t blocks = (nunits + 4 * 256 - 1) / (4 * 256);
    if (blocks < 1) blocks = 1;
    if (blocks > 16384) blocks = 16384;
    const char *s = (const char *)src;
    char *d = (char *)dst;
    void *kargs[] = {&s, &d, (void *)&nunits, (void *)&tail};
    return hipLaunchKernel((const void *)dev::copy_kernel, dim3((unsigned)blocks), dim3(256), kargs, 0,
                           (hipStream_t)stream) == hipSuccess ? AR_OK : AR_ERR_HIP;
}

int launch_bf16_round(const float *in, uint16_t *out, size_t n, void *stream)
{
    if (n == 0) return AR_OK;
    size_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    void *kargs[] = {&in, &out, &n};
    return hipLaunchKernel((const void *)dev::bf16_round_kernel, dim3((unsigned)blocks), dim3(256), kargs, 0,
                           (hipStream_t)stream) == hipSuccess ? AR_OK : AR_ERR_HIP;
}

}  // namespace ar
