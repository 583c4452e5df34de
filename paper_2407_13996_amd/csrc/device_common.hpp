// Device-side building blocks shared by the kernels of libsgdrc:
// the in-kernel CU gate, the per-CU atomic tile queues, page-table
// translation and 16-byte vector types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sgdrc {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kLutSize = 4096;          // (XCC_ID[3:0] << 8) | HW_ID[15:8]
constexpr uint32_t kLutNone = 0xFFFFFFFFu;  // key never seen by the probe
constexpr uint32_t kSkipTile = 0xFFFFFFFEu;  // a hand-back entry passed over
constexpr uint32_t kBadPage = 0xFFFFFFFFu;

constexpr uint32_t kDevErrPtRange = 1u;
constexpr uint32_t kDevFlagGateFallback = 2u;
constexpr uint32_t kDevErrSuspendedDropped = 4u;  // a suspended launch was discarded unresumed
constexpr uint32_t kDevErrHandBack = 8u;          // a handed-back tile index out of range

// Queue slot states (QueueSlot::state).
constexpr uint32_t kSlotIdle = 0u;
constexpr uint32_t kSlotSuspended = 1u;

constexpr int kMaxCus = 256;
constexpr int kMaxXcds = 16;        // XCC_ID has 4 bits
constexpr int kMaxGroups = 64;      // queue groups: runs of CUs inside one XCD
constexpr int kArrivalClasses = 8;
constexpr int kCounterStride = 32;  // 32-bit words between counters (128 bytes)
// Tiles a preemptible launch's workgroups can hand back to the resuming
// launch: at most one per workgroup per launch, so at most twice the grid
// of one launch is ever live in the ring.
constexpr uint32_t kHandBackCap = 2048;
// Partial end stamps of a statically scheduled launch's time log: 64
// addresses, so that no more than a grid / 64 workgroups meet on one.
constexpr int kTimePartials = 64;

// Work distribution state of one stream.  The CUs of each XCD are cut into
// runs of 2^grp_shift CUs ("queue groups"; a launch picks the run length:
// a whole XCD for long streaming kernels, a few CUs for short ones).  Tiles
// are split into contiguous ranges, one per group in proportion to the
// group's allowed CUs; the workgroups resident on a group's CUs claim that
// range in order through the group's ticket counter, which balances load
// dynamically inside a group while the ticket atomics spread over many
// counters.
// Arrivals are counted per class blockIdx % 8 (class sizes are known) and
// then once per class, so that the last workgroup of the grid can be found
// without every workgroup hitting one address.  That workgroup finishes any
// range that no workgroup took and zeroes the slot for the next launch on
// the stream.
//
// Preemptible launches (see gated_tile_loop) use more words: the slot's
// state (kSlotIdle, or kSlotSuspended while an evicted launch still has
// tiles to do, whose group counters are then kept for the resuming launch),
// a mark set by every workgroup that stopped on the eviction flag, a word
// that stays zero (the flag of a preemptible launch that has none), and a
// ring of tiles handed back: entries [hb_take, hb_count) (indices modulo
// kHandBackCap) wait for a resuming launch, which may claim those below
// hb_limit.
struct QueueSlot {
    uint32_t grp_next[kMaxGroups * kCounterStride];
    uint32_t done[kArrivalClasses * kCounterStride];
    uint32_t done_all[kCounterStride];
    uint32_t state[kCounterStride];
    uint32_t stopped[kCounterStride];
    uint32_t zero[kCounterStride];
    uint32_t hb_count[kCounterStride];
    uint32_t hb_take[kCounterStride];
    uint32_t hb_limit[kCounterStride];
    uint32_t hb[kHandBackCap];
    // statically scheduled launches with a time log: the latest end stamp
    // of the workgroups whose index is i mod kTimePartials, one per 128 bytes
    uint64_t tpart[kTimePartials * kCounterStride / 2];
};

// Per-launch gate arguments (passed by value in the kernel arguments).
struct Gate {
    uint64_t mask[4];            // logical CUs allowed to work
    const uint32_t *lut;         // hardware key -> logical CU | XCD << 16 | CU-in-XCD << 24
    QueueSlot *q;                // this stream's work distribution state
    uint32_t *err;               // device error / event flags
    uint32_t *log_cu;            // optional: tiles per logical CU
    uint32_t *log_tile;          // optional: visits per tile
    uint64_t log_cap;            // entries of log_tile
    uint64_t *tlog;              // optional: {start, end} wall-clock ticks of this launch
    uint32_t grp_tile[kMaxGroups + 1];  // first tile of each group's range
    uint8_t grp_base[kMaxXcds];  // first queue group of each XCD
    uint32_t n_groups;
    uint32_t grp_shift;          // log2 of CUs per queue group
    uint32_t xcc_allowed;        // bit x: XCC_ID x has allowed CUs
    const uint32_t *evict;       // preemptible launches: eviction flag (non-zero = stop)
    uint32_t resume;             // preemptible launches: 1 = continue a suspended launch
    uint32_t evict_at;           // preemptible launches, testing aid: the flag counts as
                                 // raised for tiles at or beyond this index (0 = off)
    // Static schedule (statics = 1; masks made of whole XCDs, see
    // static_tile_loop): the rank of each XCC_ID among the allowed XCDs
    // (0xFF = not allowed), their number, and the device's XCD count.
    uint32_t statics;
    uint8_t xcd_rank[kMaxXcds];
    uint32_t n_allowed_xcd;
    uint32_t n_xcd;
};

// The testing aid of preemptible launches: whether tile ``tile`` is to be
// treated as if the eviction flag had risen before it (a plain compare).
__device__ __forceinline__ uint32_t evict_hook(const Gate &g, uint32_t tile)
{
    return (g.evict_at != 0u && tile >= g.evict_at) ? 1u : 0u;
}

__device__ __forceinline__ uint32_t hw_key()
{
    uint32_t hw, xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    return ((xcc & 0xFu) << 8) | ((hw >> 8) & 0xFFu);
}

// LUT entry of the executing workgroup's CU: logical CU | XCD << 16 |
// CU-in-XCD << 24, or kLutNone.
__device__ __forceinline__ uint32_t my_cu_entry(const Gate &g)
{
    // (A vector load: reading the table as constant memory, which makes the
    // lookup a scalar load, measured 10 percent slower on the GEMV.)
    return g.lut[hw_key()];
}

__device__ __forceinline__ bool cu_allowed(const Gate &g, uint32_t cu)
{
    if (cu >= (uint32_t)kMaxCus)
        return false;
    return ((g.mask[cu >> 6] >> (cu & 63u)) & 1ull) != 0ull;
}

__device__ __forceinline__ void raise_flag(uint32_t *err, uint32_t bit)
{
    __hip_atomic_fetch_or(err, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Next ticket of a counter for the whole workgroup (thread 0 takes it).
__device__ __forceinline__ uint32_t claim_ticket(uint32_t *ctr, uint32_t *s_ticket)
{
    if (threadIdx.x == 0)
        *s_ticket = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    // the ticket is the same in every lane; make that visible to the
    // compiler so tile bases and page-table reads stay scalar
    const uint32_t t = __builtin_amdgcn_readfirstlane(*s_ticket);
    __syncthreads();
    return t;
}

// Preemptible launches, one thread: hands tile ``tile`` (claimed, not
// processed) back to the resuming launch.
__device__ __forceinline__ void hand_back(QueueSlot *q, uint32_t tile)
{
    const uint32_t i = __hip_atomic_fetch_add(&q->hb_count[0], 1u, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&q->hb[i % kHandBackCap], tile, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void log_tile(const Gate &g, uint32_t cu, uint32_t tile)
{
    if (threadIdx.x == 0) {
        if (g.log_cu && cu < (uint32_t)kMaxCus)
            __hip_atomic_fetch_add(&g.log_cu[cu], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (g.log_tile && tile < g.log_cap)
            __hip_atomic_fetch_add(&g.log_tile[tile], 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Workgroup arrival after its tile loop.  Returns true (to every thread of
// the workgroup) for the last workgroup of the grid to arrive; every
// workgroup arrives after its last ticket, so that one sees the final
// state of all counters.
//
// Ordering: every wave first waits for all of its memory operations to
// complete (the barrier alone only waits for LDS), so the workgroup's
// ticket and histogram atomics are done before the arrival atomic is
// issued; the last workgroup reads the counters with device-scope atomic
// loads issued after its arrival atomic has returned.  All of these are
// device-scope atomics, coherent across XCDs by themselves, so no fence is
// used: on gfx950 a device-scope fence writes back and invalidates the
// whole L2 of the XCD.
__device__ __forceinline__ bool arrive_last(const Gate &g, uint32_t *s_flag)
{
    __builtin_amdgcn_s_waitcnt(0);  // vmcnt, expcnt and lgkmcnt all zero
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t G = gridDim.x;
        const uint32_t grp = blockIdx.x % (uint32_t)kArrivalClasses;
        const uint32_t expected = G / kArrivalClasses + (grp < G % kArrivalClasses ? 1u : 0u);
        const uint32_t classes = G < (uint32_t)kArrivalClasses ? G : (uint32_t)kArrivalClasses;
        uint32_t last = 0u;
        const uint32_t d = __hip_atomic_fetch_add(&g.q->done[grp * kCounterStride], 1u,
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (d == expected - 1u) {
            const uint32_t e = __hip_atomic_fetch_add(&g.q->done_all[0], 1u, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT);
            last = e == classes - 1u ? 1u : 0u;
        }
        *s_flag = last;
    }
    __syncthreads();
    return *s_flag != 0u;
}

// Called by the last workgroup only, after all its work: zero the slot
// (the group counters too unless ``keep_counters``, which leaves them to a
// resuming launch).
__device__ __forceinline__ void reset_slot(QueueSlot *q, bool keep_counters = false)
{
    __syncthreads();
    if (!keep_counters && threadIdx.x < (uint32_t)kMaxGroups)
        __hip_atomic_store(&q->grp_next[threadIdx.x * kCounterStride], 0u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x < (uint32_t)kArrivalClasses)
        __hip_atomic_store(&q->done[threadIdx.x * kCounterStride], 0u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0)
        __hip_atomic_store(&q->done_all[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct NoOp {
    __device__ void operator()() const {}
};

// When a workgroup takes its next ticket relative to the work of a tile.
//  Ahead: before the tile, so that the round trip overlaps the whole tile;
//    pays off for short launches of one or two tiles per workgroup (GEMV).
//  Mid:   where the body calls ``claim()``: streaming bodies call it after
//    issuing their loads and before their stores.  On gfx950 one counter
//    tracks loads, stores and atomics of a wave in issue order, so waiting
//    for a ticket taken after the stores also waits for the stores to be
//    acknowledged by memory, and a ticket taken before the loads holds the
//    loads back behind a contended atomic; between the two it costs neither.
//  After: after the tile.
enum class Claim { Ahead, Mid, After };

// Runs ``prologue()`` once at the start, alongside the gate's own reads and
// before a barrier (kernels stage per-launch tables there; it should be
// straight-line code), then ``body(tile, cu, err, claim)`` for every tile
// that this workgroup obtains, under the gate.  Workgroups on CUs outside the mask take no
// tiles; the others take tiles of their own group's range, then steal from
// other groups' ranges until every range is exhausted.  ``flush()`` runs
// after a workgroup's tile loop (to publish per-workgroup partials).  The
// last workgroup to arrive finishes the tiles of any range that no
// workgroup took (only possible when no workgroup landed on any allowed CU;
// flagged), flushes again, calls ``epilogue()`` with every other
// workgroup's work complete, and zeroes the slot.
//
// ``claim`` is a callable that every thread of the workgroup calls exactly
// once per tile, on a workgroup-uniform path; only Claim::Mid gives it an
// effect.
//
// Preemptible launches (EV, Claim::Mid only): a workgroup reads the
// eviction flag ``*g.evict`` at its start, at the start of each tile and
// right after each claim.  Once it has seen the flag set it takes no more
// tickets: it finishes the tile it is working on and leaves, and marks the
// slot; a ticket it claimed before the flag rose is handed back (its tile
// goes to the slot's hand-back ring) rather than worked on, so that the
// workgroup leaves after one tile, not two.
// If tiles are left (unclaimed or handed back) when the last workgroup
// arrives and some workgroup stopped on the flag, the launch is suspended
// instead of completed: the last workgroup leaves the remaining tiles and
// the epilogue alone, keeps the group counters and the ring, and sets the
// slot's state to kSlotSuspended.  A resuming launch (``g.resume``, same
// kernel arguments and tile ranges, any mask) first works through the
// handed-back tiles, then continues from the group counters, stealing
// across groups as usual, and does nothing if the slot is idle (the launch
// it resumes had completed).  Fresh launches start on an idle slot (the
// host discards a suspended launch first, see k_slot_discard).
//
// Bodies must not return early or branch around the rest of the tile on a
// per-lane condition: the loop contains barriers, and a lane-dependent exit
// from it lets the compiler send some lanes of a wave back to the barrier
// while others still owe the next ticket.  Bodies record problems in the
// per-thread ``err`` bits instead; they are raised once, after the loop.
template <Claim CL, bool EV = false, typename Prologue, typename Body, typename Flush,
          typename Epilogue>
__device__ __forceinline__ void gated_tile_loop(const Gate &g, uint32_t n_tiles, Prologue prologue,
                                                Body body, Flush flush, Epilogue epilogue)
{
    static_assert(!EV || CL == Claim::Mid, "preemptible launches claim mid-tile");
    __shared__ uint32_t s_ticket;
    __shared__ uint32_t s_stop;
    __shared__ uint32_t s_flag;
    __shared__ uint32_t s_left_lo[kMaxGroups], s_left_hi[kMaxGroups];
    __shared__ uint32_t s_grp_tile[kMaxGroups + 1];
    __shared__ uint32_t s_hb_lo, s_hb_hi;
    // Prologue: every memory read it needs is issued before any branch on
    // a value read, so that the round trips overlap (the CU-table entry is
    // read even on an XCD without allowed CUs, and then ignored).
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const uint32_t lut_entry = my_cu_entry(g);
    // preemptible: thread 0 reads the slot state and the flag; both reach
    // the other threads through LDS, so the whole workgroup decides alike
    // even if the flag changes meanwhile
    uint32_t slot_state = 0u, flag0 = 0u;
    if (EV && threadIdx.x == 0) {
        slot_state = __hip_atomic_load(&g.q->state[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        flag0 = __hip_atomic_load(g.evict, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // every kernel runs at least kMaxGroups + 1 threads per workgroup; the
    // threads beyond write the last entry again (same value), which keeps
    // this straight-line code
    {
        const uint32_t i = threadIdx.x < (uint32_t)kMaxGroups ? threadIdx.x : (uint32_t)kMaxGroups;
        s_grp_tile[i] = g.grp_tile[i];
    }
    prologue();
    const bool xcd_on = ((g.xcc_allowed >> (xcc & 0xFu)) & 1u) != 0u;
    const uint32_t entry = xcd_on ? lut_entry : kLutNone;
    if (EV && threadIdx.x == 0) {
        // a launch with nothing to do: a resume of a completed launch
        s_flag = (g.resume && slot_state != kSlotSuspended) ? 1u : 0u;
        s_stop = flag0 != 0u ? 1u : 0u;
    }
    // time log: workgroup 0, the first one the hardware dispatches, stamps
    // the start; the last workgroup to finish stamps the end
    if (g.tlog && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(&g.tlog[0], __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const bool dead = EV && __builtin_amdgcn_readfirstlane(s_flag) != 0u;
    const bool stop0 = EV && __builtin_amdgcn_readfirstlane(s_stop) != 0u;
    // s_flag and s_stop are written again only after the barriers that
    // follow (arrival, first ticket or first tile)
    uint32_t err = 0u;
    const uint32_t cu = entry & 0xFFFFu;
    if (!dead && entry != kLutNone && cu_allowed(g, cu)) {
        uint32_t grp = g.grp_base[(entry >> 16) & 0xFFu] + ((entry >> 24) >> g.grp_shift);
        uint32_t lo = s_grp_tile[grp], hi = s_grp_tile[grp + 1u];
        // preemptible: a workgroup that sees the flag at its start takes no
        // ticket at all
        bool stop = stop0;
        if (EV && g.resume) {
            // a resuming launch first works through the tiles handed back by
            // the launch it resumes, claiming them one at a time; a claimed
            // one goes back to the ring if the flag is up again.  (The
            // barrier: every wave has read s_stop before it is reused.)
            __syncthreads();
            for (;;) {
                if (threadIdx.x == 0) {
                    uint32_t tile = kLutNone, fl = 0u;
                    if (!stop) {
                        const uint32_t lim = __hip_atomic_load(&g.q->hb_limit[0], __ATOMIC_RELAXED,
                                                               __HIP_MEMORY_SCOPE_AGENT);
                        const uint32_t i = __hip_atomic_fetch_add(&g.q->hb_take[0], 1u,
                                                                  __ATOMIC_RELAXED,
                                                                  __HIP_MEMORY_SCOPE_AGENT);
                        fl = __hip_atomic_load(g.evict, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if (i < lim) {
                            tile = __hip_atomic_load(&g.q->hb[i % kHandBackCap], __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
                            fl |= evict_hook(g, tile);
                            if (tile >= n_tiles) {
                                // never expected: skip the entry, keep draining
                                err |= kDevErrHandBack;
                                tile = kSkipTile;
                            } else if (fl != 0u) {
                                hand_back(g.q, tile);
                                tile = kLutNone;
                            }
                        }
                    }
                    s_ticket = tile;
                    s_stop = (stop || fl != 0u) ? 1u : 0u;
                }
                __syncthreads();
                const uint32_t tile = __builtin_amdgcn_readfirstlane(s_ticket);
                stop = __builtin_amdgcn_readfirstlane(s_stop) != 0u;
                __syncthreads();
                if (tile == kLutNone)
                    break;
                if (tile != kSkipTile) {
                    log_tile(g, cu, tile);
                    body(tile, cu, err, NoOp());
                }
            }
        }
        uint32_t k = stop ? kLutNone : claim_ticket(&g.q->grp_next[grp * kCounterStride], &s_ticket);
        // One flat loop: work through the own group's range, then steal from
        // the next group in ring order that still has tiles, found by wave 0
        // reading every group's counter at once.
        //
        // ``next`` lives across iterations and is written only by the ticket
        // atomic: re-initialising it in the loop would be a vector-ALU write
        // to the atomic's destination register, for which the compiler waits
        // on the memory counter, stalling the tile's loads behind the
        // previous tile's stores.
        uint32_t next = 0u, fl2 = 0u;
        for (;;) {
            if (k < hi - lo) {
                uint32_t *const ctr = &g.q->grp_next[grp * kCounterStride];
                // preemptible: the flag is read before the tile's loads, so
                // that its value is back when the next ticket is claimed; once
                // it is set, the claim adds 0 (no branch around the atomic)
                // and this tile is the workgroup's last
                uint32_t fl = 0u;
                if (EV && threadIdx.x == 0)
                    fl = __hip_atomic_load(g.evict, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) |
                         evict_hook(g, lo + k);
                if (CL == Claim::Ahead && threadIdx.x == 0)
                    next = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                auto claim = [&]() {
                    if (CL == Claim::Mid && threadIdx.x == 0) {
                        next = __hip_atomic_fetch_add(ctr, (EV && fl != 0u) ? 0u : 1u,
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        // preemptible: the flag again, issued before the
                        // stores, so its value is back with the ticket
                        if (EV)
                            fl2 = __hip_atomic_load(g.evict, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
                    }
                };
                log_tile(g, cu, lo + k);
                body(lo + k, cu, err, claim);
                if (CL == Claim::After && threadIdx.x == 0)
                    next = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (threadIdx.x == 0) {
                    // halt: the claim added nothing (flag seen at the tile's
                    // start); late: the flag rose after that, so the ticket
                    // just claimed is handed back instead of worked on
                    const bool halt = EV && fl != 0u;
                    const bool late = EV && !halt && (fl2 | evict_hook(g, lo + next)) != 0u;
                    if (late && next < hi - lo)
                        hand_back(g.q, lo + next);
                    s_ticket = (halt || late) ? kLutNone : next;
                    if (EV)
                        s_stop = (halt || late) ? 1u : 0u;
                }
                __syncthreads();
                k = __builtin_amdgcn_readfirstlane(s_ticket);
                if (EV)
                    stop = __builtin_amdgcn_readfirstlane(s_stop) != 0u;
                __syncthreads();
            } else {
                if (EV && stop)
                    break;
                if (threadIdx.x < 64u) {
                    const uint32_t r = threadIdx.x;
                    bool rem = false;
                    if (r < g.n_groups) {
                        const uint32_t size = s_grp_tile[r + 1u] - s_grp_tile[r];
                        const uint32_t taken =
                            size ? __hip_atomic_load(&g.q->grp_next[r * kCounterStride],
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                 : 0u;
                        rem = taken < size;
                    }
                    uint32_t fl = 0u;
                    if (EV && r == 0u)
                        fl = __hip_atomic_load(g.evict, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    const uint64_t bits = __ballot(rem);
                    if (threadIdx.x == 0) {
                        uint32_t pick = kLutNone;
                        if (bits) {
                            const uint32_t sh = (grp + 1u) & 63u;
                            const uint64_t rot = sh ? ((bits >> sh) | (bits << (64u - sh))) : bits;
                            pick = (sh + (uint32_t)__builtin_ctzll(rot)) & 63u;
                        }
                        s_ticket = pick;
                        if (EV)
                            s_stop = fl != 0u ? 1u : 0u;
                    }
                }
                __syncthreads();
                const uint32_t pick = __builtin_amdgcn_readfirstlane(s_ticket);
                if (EV)
                    stop = __builtin_amdgcn_readfirstlane(s_stop) != 0u;
                __syncthreads();
                if (pick == kLutNone || (EV && stop))
                    break;
                grp = pick;
                lo = s_grp_tile[grp];
                hi = s_grp_tile[grp + 1u];
                k = claim_ticket(&g.q->grp_next[grp * kCounterStride], &s_ticket);
            }
        }
        if (EV && stop && threadIdx.x == 0)
            __hip_atomic_store(&g.q->stopped[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        flush();
    }
    if (arrive_last(g, &s_flag)) {
        // ranges that no workgroup finished: [lo + tickets taken, hi)
        bool left = false;
        if (threadIdx.x < (uint32_t)kMaxGroups) {
            uint32_t a = 0u, b = 0u;
            if (threadIdx.x < g.n_groups) {
                const uint32_t lo = g.grp_tile[threadIdx.x], hi = g.grp_tile[threadIdx.x + 1u];
                const uint32_t taken = __hip_atomic_load(&g.q->grp_next[threadIdx.x * kCounterStride],
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                a = taken < hi - lo ? lo + taken : hi;
                b = hi;
            }
            s_left_lo[threadIdx.x] = a;
            s_left_hi[threadIdx.x] = b;
            left = a < b;
        }
        if (threadIdx.x == 0) {
            s_stop = EV ? __hip_atomic_load(&g.q->stopped[0], __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT)
                        : 0u;
            if (EV) {
                // handed-back tiles not yet worked on: [min(take, limit), count)
                const uint32_t cnt = __hip_atomic_load(&g.q->hb_count[0], __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t take = __hip_atomic_load(&g.q->hb_take[0], __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t lim = __hip_atomic_load(&g.q->hb_limit[0], __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t from = take < lim ? take : lim;
                s_hb_lo = from;
                s_hb_hi = cnt;
                left = left || from < cnt;
            }
        }
        const bool any_left = __syncthreads_or(left ? 1 : 0) != 0;
        const bool stopped = EV && __builtin_amdgcn_readfirstlane(s_stop) != 0u;
        if (EV && dead) {
            // nothing ran: only the arrival counters are reset
            reset_slot(g.q, true);
        } else if (EV && any_left && stopped) {
            // suspended: the unclaimed and handed-back tiles wait for a
            // resuming launch, which may claim the ring up to its end now
            reset_slot(g.q, true);
            if (threadIdx.x == 0) {
                __hip_atomic_store(&g.q->hb_take[0], s_hb_lo, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->hb_limit[0], s_hb_hi, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->stopped[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->state[0], kSlotSuspended, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
        } else {
            if (any_left) {
                if (EV) {
                    // handed-back tiles that no workgroup took (none reached
                    // an allowed CU)
                    uint32_t i = __builtin_amdgcn_readfirstlane(s_hb_lo);
                    const uint32_t e = __builtin_amdgcn_readfirstlane(s_hb_hi);
                    while (i < e) {
                        const uint32_t t = __builtin_amdgcn_readfirstlane(__hip_atomic_load(
                            &g.q->hb[i % kHandBackCap], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                        if (t < n_tiles) {
                            log_tile(g, cu, t);
                            body(t, cu, err, NoOp());
                        } else {
                            err |= threadIdx.x == 0 ? kDevErrHandBack : 0u;
                        }
                        i += 1u;
                    }
                }
                // worked through in one flat loop so that no barrier of the
                // body ends up in a nested loop
                uint32_t c = 0u;
                uint32_t t = __builtin_amdgcn_readfirstlane(s_left_lo[0]);
                uint32_t end = __builtin_amdgcn_readfirstlane(s_left_hi[0]);
                while (c < (uint32_t)kMaxGroups) {
                    if (t < end) {
                        log_tile(g, cu, t);
                        body(t, cu, err, NoOp());
                        t += 1u;
                    } else {
                        c += 1u;
                        const uint32_t cc = c < (uint32_t)kMaxGroups ? c : 0u;
                        t = __builtin_amdgcn_readfirstlane(s_left_lo[cc]);
                        end = c < (uint32_t)kMaxGroups ? __builtin_amdgcn_readfirstlane(s_left_hi[cc]) : 0u;
                    }
                }
                flush();
                err |= threadIdx.x == 0 ? kDevFlagGateFallback : 0u;
            }
            __builtin_amdgcn_s_waitcnt(0);  // own partials complete before the epilogue reads
            __syncthreads();
            epilogue();
            reset_slot(g.q);
            if (EV && threadIdx.x == 0) {
                __hip_atomic_store(&g.q->stopped[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->hb_count[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->hb_take[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->hb_limit[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&g.q->state[0], kSlotIdle, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        if (g.tlog && threadIdx.x == 0) {
            __builtin_amdgcn_s_waitcnt(0);
            __hip_atomic_store(&g.tlog[1], __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (err != 0u)
        raise_flag(g.err, err);
}

// Static schedule for launches whose CU mask is a union of whole XCDs (the
// host sets g.statics).  The hardware hands the workgroups of a grid to the
// XCDs by index modulo the XCD count (checked at context creation), so a
// workgroup knows its XCD from XCC_ID and its rank among the workgroups of
// that XCD from blockIdx alone: no table lookup, no ticket, no arrival
// counter.  With A allowed XCDs and W workgroups per XCD, the workgroup of
// rank r on the allowed XCD of rank a is worker v = r A + a of W A, and
// takes tiles v, v + W A, ... -- consecutive tiles on different XCDs, as a
// plain grid would place them.  Workgroups on other XCDs leave at once.
// With a time log, workgroup 0 stamps the start and every workgroup, once
// its stores are done, raises partial end stamp blockIdx mod kTimePartials
// to its end time; the host reduces the partials with k_tlog_reduce after
// the launch.  ``prologue`` and ``body`` as in gated_tile_loop (``claim`` has
// no effect).
template <typename Prologue, typename Body>
__device__ __forceinline__ void static_tile_loop(const Gate &g, uint32_t n_tiles, Prologue prologue,
                                                 Body body)
{
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const uint32_t a = g.xcd_rank[xcc & 0xFu];
    // the work log names the logical CU: one table read, only when logging
    const uint32_t cu = g.log_cu ? (my_cu_entry(g) & 0xFFFFu) : (uint32_t)kMaxCus;
    prologue();
    if (g.tlog && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(&g.tlog[0], __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    uint32_t err = 0u;
    if (a != 0xFFu) {
        const uint32_t workers = (gridDim.x / g.n_xcd) * g.n_allowed_xcd;
        for (uint32_t t = (blockIdx.x / g.n_xcd) * g.n_allowed_xcd + a; t < n_tiles; t += workers) {
            log_tile(g, cu, t);
            body(t, cu, err, NoOp());
        }
    }
    if (g.tlog) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0)
            __hip_atomic_fetch_max(&g.q->tpart[(blockIdx.x % kTimePartials) * (kCounterStride / 2)],
                                   (uint64_t)__builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
    if (err != 0u)
        raise_flag(g.err, err);
}

// The gate's two schedules behind one call: static for masks of whole XCDs
// (g.statics, a uniform branch), the ticket queues otherwise.
template <Claim CL, typename Prologue, typename Body>
__device__ __forceinline__ void tile_loop(const Gate &g, uint32_t n_tiles, Prologue prologue, Body body)
{
    if (g.statics)
        static_tile_loop(g, n_tiles, prologue, body);
    else
        gated_tile_loop<CL>(g, n_tiles, prologue, body, NoOp(), NoOp());
}

// Wavefront-granular form of gated_tile_loop, for bodies whose work is
// private to one wavefront (they share no LDS between the waves of a
// workgroup and contain no barrier).  Each wavefront takes its own tickets
// (lane 0 runs the atomic, the value reaches the other lanes by
// readfirstlane), so the loop holds no barrier: the waves of a workgroup
// drift apart and keep loads in flight while a neighbour finishes a tile,
// instead of draining the memory pipe together at every tile.  ``claim`` has
// the Claim::Mid meaning.  Gate, queue groups, stealing, ``flush`` (per
// workgroup, after all of its waves leave the loop), the last workgroup's
// leftover ranges (spread over its waves) and ``epilogue`` are as in
// gated_tile_loop.
__device__ __forceinline__ void log_tile_wave(const Gate &g, uint32_t cu, uint32_t tile)
{
    if ((threadIdx.x & 63u) == 0u) {
        if (g.log_cu && cu < (uint32_t)kMaxCus)
            __hip_atomic_fetch_add(&g.log_cu[cu], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (g.log_tile && tile < g.log_cap)
            __hip_atomic_fetch_add(&g.log_tile[tile], 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <typename Prologue, typename Body, typename Flush, typename Epilogue>
__device__ __forceinline__ void gated_wave_loop(const Gate &g, uint32_t n_tiles, Prologue prologue,
                                                Body body, Flush flush, Epilogue epilogue)
{
    __shared__ uint32_t s_flag;
    __shared__ uint32_t s_left_lo[kMaxGroups], s_left_hi[kMaxGroups];
    __shared__ uint32_t s_grp_tile[kMaxGroups + 1];
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const uint32_t lut_entry = my_cu_entry(g);
    {
        const uint32_t i = threadIdx.x < (uint32_t)kMaxGroups ? threadIdx.x : (uint32_t)kMaxGroups;
        s_grp_tile[i] = g.grp_tile[i];
    }
    prologue();
    const bool xcd_on = ((g.xcc_allowed >> (xcc & 0xFu)) & 1u) != 0u;
    const uint32_t entry = xcd_on ? lut_entry : kLutNone;
    if (g.tlog && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(&g.tlog[0], __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    uint32_t err = 0u;
    const uint32_t cu = entry & 0xFFFFu;
    const uint32_t lane = threadIdx.x & 63u;
    if (entry != kLutNone && cu_allowed(g, cu)) {
        uint32_t grp = g.grp_base[(entry >> 16) & 0xFFu] + ((entry >> 24) >> g.grp_shift);
        uint32_t lo = s_grp_tile[grp], hi = s_grp_tile[grp + 1u];
        // ``next`` holds the ticket in lane 0; written only by the atomic
        // (see gated_tile_loop)
        uint32_t next = 0u;
        if (lane == 0u)
            next = __hip_atomic_fetch_add(&g.q->grp_next[grp * kCounterStride], 1u,
                                          __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        uint32_t k = __builtin_amdgcn_readfirstlane(next);
        for (;;) {
            if (k < hi - lo) {
                uint32_t *const ctr = &g.q->grp_next[grp * kCounterStride];
                auto claim = [&]() {
                    if (lane == 0u)
                        next = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT);
                };
                log_tile_wave(g, cu, lo + k);
                body(lo + k, cu, err, claim);
                k = __builtin_amdgcn_readfirstlane(next);
            } else {
                // steal: the next group in ring order that still has tiles
                bool rem = false;
                if (lane < g.n_groups) {
                    const uint32_t size = s_grp_tile[lane + 1u] - s_grp_tile[lane];
                    const uint32_t taken =
                        size ? __hip_atomic_load(&g.q->grp_next[lane * kCounterStride],
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                             : 0u;
                    rem = taken < size;
                }
                const uint64_t bits = __ballot(rem);
                if (bits == 0ull)
                    break;
                const uint32_t sh = (grp + 1u) & 63u;
                const uint64_t rot = sh ? ((bits >> sh) | (bits << (64u - sh))) : bits;
                grp = __builtin_amdgcn_readfirstlane((sh + (uint32_t)__builtin_ctzll(rot)) & 63u);
                lo = s_grp_tile[grp];
                hi = s_grp_tile[grp + 1u];
                if (lane == 0u)
                    next = __hip_atomic_fetch_add(&g.q->grp_next[grp * kCounterStride], 1u,
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                k = __builtin_amdgcn_readfirstlane(next);
            }
        }
        flush();
    }
    if (arrive_last(g, &s_flag)) {
        bool left = false;
        if (threadIdx.x < (uint32_t)kMaxGroups) {
            uint32_t a = 0u, b = 0u;
            if (threadIdx.x < g.n_groups) {
                const uint32_t lo = g.grp_tile[threadIdx.x], hi = g.grp_tile[threadIdx.x + 1u];
                const uint32_t taken = __hip_atomic_load(&g.q->grp_next[threadIdx.x * kCounterStride],
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                a = taken < hi - lo ? lo + taken : hi;
                b = hi;
            }
            s_left_lo[threadIdx.x] = a;
            s_left_hi[threadIdx.x] = b;
            left = a < b;
        }
        if (__syncthreads_or(left ? 1 : 0)) {
            // wave w takes tiles lo + w, lo + w + waves, ... of each range
            const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
            const uint32_t waves = blockDim.x >> 6;
            uint32_t c = 0u;
            uint32_t t = __builtin_amdgcn_readfirstlane(s_left_lo[0]) + wave;
            uint32_t end = __builtin_amdgcn_readfirstlane(s_left_hi[0]);
            while (c < (uint32_t)kMaxGroups) {
                if (t < end) {
                    log_tile_wave(g, cu, t);
                    body(t, cu, err, NoOp());
                    t += waves;
                } else {
                    c += 1u;
                    const uint32_t cc = c < (uint32_t)kMaxGroups ? c : 0u;
                    t = __builtin_amdgcn_readfirstlane(s_left_lo[cc]) + wave;
                    end = c < (uint32_t)kMaxGroups ? __builtin_amdgcn_readfirstlane(s_left_hi[cc]) : 0u;
                }
            }
            flush();
            err |= threadIdx.x == 0 ? kDevFlagGateFallback : 0u;
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        epilogue();
        reset_slot(g.q);
        if (g.tlog && threadIdx.x == 0) {
            __builtin_amdgcn_s_waitcnt(0);
            __hip_atomic_store(&g.tlog[1], __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (err != 0u)
        raise_flag(g.err, err);
}

// Static form of gated_wave_loop, for masks made of whole XCDs (g.statics,
// as static_tile_loop): the workers are the wavefronts, numbered so that the
// waves of one workgroup take consecutive tiles, and wave v of the W
// workers takes tiles v, v + W, ...  ``flush`` runs once the workgroup's
// waves are done; there is no last workgroup, so no epilogue: the host
// enqueues whatever must follow the whole grid as a kernel of its own.
template <typename Prologue, typename Body, typename Flush>
__device__ __forceinline__ void static_wave_loop(const Gate &g, uint32_t n_tiles, Prologue prologue,
                                                 Body body, Flush flush)
{
    uint32_t xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const uint32_t a = g.xcd_rank[xcc & 0xFu];
    const uint32_t cu = g.log_cu ? (my_cu_entry(g) & 0xFFFFu) : (uint32_t)kMaxCus;
    prologue();
    if (g.tlog && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(&g.tlog[0], __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    uint32_t err = 0u;
    if (a != 0xFFu) {
        const uint32_t waves = blockDim.x >> 6;
        const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const uint32_t workers = (gridDim.x / g.n_xcd) * g.n_allowed_xcd * waves;
        for (uint32_t t = ((blockIdx.x / g.n_xcd) * g.n_allowed_xcd + a) * waves + wave; t < n_tiles;
             t += workers) {
            log_tile_wave(g, cu, t);
            body(t, cu, err, NoOp());
        }
        flush();
    }
    if (g.tlog) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0)
            __hip_atomic_fetch_max(&g.q->tpart[(blockIdx.x % kTimePartials) * (kCounterStride / 2)],
                                   (uint64_t)__builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
    if (err != 0u)
        raise_flag(g.err, err);
}

// Page-table lookup with the range check every kernel applies: an entry
// outside the pool yields kBadPage and sets kDevErrPtRange in ``err``.
__device__ __forceinline__ uint32_t checked_page(const uint32_t *pt, uint64_t j,
                                                 uint64_t pool_pages, uint32_t &err)
{
    const uint32_t p = pt[j];
    const bool bad = (uint64_t)p >= pool_pages;
    err |= bad ? kDevErrPtRange : 0u;
    return bad ? kBadPage : p;
}

// Buffer resources (gfx9 descriptor, raw addressing: stride 0, byte offsets,
// data-format word as used for untyped buffers on this family).  Accesses at
// byte offsets at or beyond ``bytes`` are dropped by the hardware: loads
// return zero and stores write nothing.  Kernels keep every 16-byte access
// 16-byte aligned and every range a multiple of 16 bytes, so an access is
// either wholly inside or wholly outside its range.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;
constexpr int kAuxNt = 2;  // cache policy: non-temporal
// Streaming stores: non-temporal and SC1 (written through past the L2 rather
// than left dirty in it); measured 1.5-2.5 percent faster than non-temporal
// alone for the triad and the relayout on MI355X, SC1 alone no faster.
constexpr int kAuxStore = 16 | kAuxNt;
// Classify's colour stores: SC1 without the non-temporal bit.  Its stores
// are one byte per eight bytes read, and with NT they cost 5-6 percent of
// the kernel (2^26 addresses on MI355X: 102.3 against 96.7 us, with
// histogram 105 against 99; SC0+SC1 the same as SC1, cached stores or NT
// alone 98.7-98.8 us).
constexpr int kAuxStoreSc1 = 16;

__device__ __forceinline__ Rsrc make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             kRsrcWord3);
}

__device__ __forceinline__ u32x4 buf_load_nt(Rsrc r, uint32_t off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kAuxNt));
}

__device__ __forceinline__ void buf_store_nt(Rsrc r, uint32_t off, u32x4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), r, off, 0, kAuxStore);
}

__device__ __forceinline__ void buf_store_sc1(Rsrc r, uint32_t off, u32x4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), r, off, 0, kAuxStoreSc1);
}

__device__ __forceinline__ u32x4 load_nt(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ void store_nt(void *p, u32x4 v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p));
}

}  // namespace sgdrc
