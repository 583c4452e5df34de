// Device-side building blocks shared by the kernels of libsgdrc:
// the in-kernel CU gate, the self-resetting atomic tile queue, page-table
// translation and 16-byte vector types.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sgdrc {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

constexpr int kLutSize = 4096;          // (XCC_ID[3:0] << 8) | HW_ID[15:8]
constexpr uint16_t kLutNone = 0xFFFFu;  // key never seen by the probe
constexpr uint32_t kBadPage = 0xFFFFFFFFu;

constexpr uint32_t kDevErrPtRange = 1u;
constexpr uint32_t kDevFlagGateFallback = 2u;

// One work queue per stream.  ``next`` hands out tile indices; ``done``
// counts finished workgroups so that the last one can reset both, which
// leaves the queue at zero for the next launch on the same stream.
struct alignas(128) TileQueue {
    uint32_t next;
    uint32_t done;
    uint32_t pad[30];
};

// Per-launch gate arguments (passed by value in the kernel arguments).
struct Gate {
    uint64_t mask[4];         // logical CUs allowed to work
    const uint16_t *lut;      // hardware key -> logical CU
    TileQueue *q;             // this stream's queue
    uint32_t *err;            // device error / event flags
    uint32_t *log_cu;         // optional: tiles per logical CU
    uint32_t *log_tile;       // optional: visits per tile
    uint64_t log_cap;         // entries of log_tile
};

__device__ __forceinline__ uint32_t hw_key()
{
    uint32_t hw, xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID)" : "=s"(hw));
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    return ((xcc & 0xFu) << 8) | ((hw >> 8) & 0xFFu);
}

// Logical CU of the executing workgroup, or kLutNone.
__device__ __forceinline__ uint32_t my_cu(const Gate &g)
{
    return g.lut[hw_key()];
}

__device__ __forceinline__ bool cu_allowed(const Gate &g, uint32_t cu)
{
    if (cu >= 256u)
        return false;
    return ((g.mask[cu >> 6] >> (cu & 63u)) & 1ull) != 0ull;
}

__device__ __forceinline__ void raise_flag(uint32_t *err, uint32_t bit)
{
    __hip_atomic_fetch_or(err, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Claim the next tile for the whole workgroup (thread 0 takes the ticket).
__device__ __forceinline__ uint32_t claim_tile(TileQueue *q, uint32_t *s_ticket)
{
    if (threadIdx.x == 0)
        *s_ticket = __hip_atomic_fetch_add(&q->next, 1u, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    // the ticket is the same in every lane; make that visible to the
    // compiler so tile bases and page-table reads stay scalar
    uint32_t t = __builtin_amdgcn_readfirstlane(*s_ticket);
    __syncthreads();
    return t;
}

__device__ __forceinline__ void log_tile(const Gate &g, uint32_t cu, uint32_t tile)
{
    if (threadIdx.x == 0) {
        if (g.log_cu && cu < 256u)
            __hip_atomic_fetch_add(&g.log_cu[cu], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (g.log_tile && tile < g.log_cap)
            __hip_atomic_fetch_add(&g.log_tile[tile], 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Workgroup arrival at the end of its tile loop.  Returns true (to every
// thread of the workgroup) for the last workgroup of the grid to arrive.
// Every workgroup arrives after its last ticket, so the last one sees the
// final state of the queue.
__device__ __forceinline__ bool arrive_last(TileQueue *q, uint32_t *s_flag)
{
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        uint32_t d = __hip_atomic_fetch_add(&q->done, 1u, __ATOMIC_ACQ_REL,
                                            __HIP_MEMORY_SCOPE_AGENT);
        *s_flag = (d == gridDim.x - 1u) ? 1u : 0u;
    }
    __syncthreads();
    return *s_flag != 0u;
}

// Called by the last workgroup only, after all its work: zero the queue.
__device__ __forceinline__ void reset_queue(TileQueue *q)
{
    __syncthreads();
    if (threadIdx.x == 0) {
        __hip_atomic_store(&q->next, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&q->done, 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Runs ``body(tile, cu, err)`` for every tile this workgroup obtains, under
// the gate.  Workgroups on CUs outside the mask take no tiles.  ``flush()``
// runs after a workgroup's tile loop (to publish per-workgroup partials).
// The last workgroup to arrive finishes any tiles left over (possible only
// when no workgroup landed on an allowed CU; flagged), flushes again, calls
// ``epilogue()`` with every other workgroup's work complete, and resets the
// queue for the next launch on the stream.
//
// Bodies must not return early or branch around the rest of the tile on a
// per-lane condition: the loop contains barriers, and a lane-dependent exit
// from it lets the compiler send some lanes of a wave back to the barrier
// while others still owe the next ticket.  Bodies record problems in the
// per-thread ``err`` bits instead; they are raised once, after the loop.
template <typename Body, typename Flush, typename Epilogue>
__device__ __forceinline__ void gated_tile_loop(const Gate &g, uint32_t n_tiles, Body body,
                                                Flush flush, Epilogue epilogue)
{
    __shared__ uint32_t s_ticket;
    __shared__ uint32_t s_flag;
    uint32_t err = 0u;
    const uint32_t cu = my_cu(g);
    if (cu_allowed(g, cu)) {
        for (;;) {
            const uint32_t t = claim_tile(g.q, &s_ticket);
            if (t >= n_tiles)
                break;
            log_tile(g, cu, t);
            body(t, cu, err);
        }
        flush();
    }
    if (arrive_last(g.q, &s_flag)) {
        uint32_t leftover = 0u;
        for (;;) {
            const uint32_t t = claim_tile(g.q, &s_ticket);
            if (t >= n_tiles)
                break;
            leftover += 1u;
            log_tile(g, cu, t);
            body(t, cu, err);
        }
        if (leftover != 0u) {
            flush();
            err |= threadIdx.x == 0 ? kDevFlagGateFallback : 0u;
        }
        __syncthreads();
        epilogue();
        reset_queue(g.q);
    }
    if (err != 0u)
        raise_flag(g.err, err);
}

struct NoOp {
    __device__ void operator()() const {}
};

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

__device__ __forceinline__ u32x4 load_nt(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ void store_nt(void *p, u32x4 v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p));
}

}  // namespace sgdrc
