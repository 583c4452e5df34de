// Host-side internals of libsgdrc: the context, error reporting, per-stream
// state and launch sizing.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <functional>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "device_common.hpp"
#include "sgdrc.h"

namespace sgdrc {

constexpr uint32_t kCtxMagic = 0x53474452u;  // "SGDR"
constexpr int kMaxStreams = 64;
constexpr int kHistBins = 256;
// Copies of each stream's histogram accumulators in device memory: a
// workgroup adds its counts to the copy of its XCD, so that the workgroups'
// device-scope atomics spread over eight addresses per bin.
constexpr int kHistAccCopies = 8;
// CUs served by one work queue.  Long streaming kernels use one queue for
// the whole device (0): tiles are then taken in address order by all CUs
// together, which measured faster on MI355X than splitting the address range
// over per-XCD queues.  Short kernels such as the GEMV use queues of a few
// CUs, so that fewer workgroups contend on each counter.
constexpr int kStreamGroupCus = 0;
constexpr int kGemvGroupCus = 8;

// Re-issues a preemptible launch with a given gate and grid size.
typedef std::function<hipError_t(const Gate &, uint32_t grid)> Relaunch;

struct StreamState {
    int slot = -1;
    sgdrc_cu_mask mask{};
    uint32_t wg_cap = 0;        // workgroups per CU at most (0 = as many as fit)
    uint64_t last_tiles = 0;
    uint64_t *tlog = nullptr;   // time-log slots ({start, end} pairs) or NULL
    uint32_t tlog_slots = 0;
    uint64_t tlog_next = 0;     // launches logged since the log was set
    // preemptible launches: their own queue slot (so that a suspended
    // launch never meets another kernel of the stream), the eviction flag,
    // and the last such launch, kept for sgdrc_resume
    int slot_ev = -1;
    bool ev_on = false;
    const uint32_t *evict = nullptr;
    Relaunch ev_relaunch;
    Gate ev_gate{};             // tile ranges and queue-group layout of that launch
    uint64_t ev_tiles = 0;
    int ev_per_cu = 1;
    uint32_t evict_at = 0;      // testing aid: the flag counts as raised from this tile (0 = off)
    uint32_t last_schedule = 0; // schedule of the last launch: 0 ticket queues, 1 static
};

// What a gated launch needs besides the Gate itself.
struct LaunchInfo {
    int allowed = 0;            // allowed CUs
    uint32_t wg_cap = 0;        // per-stream cap on workgroups per CU
};

struct Ctx {
    uint32_t magic = kCtxMagic;
    int device = -1;
    int num_cus = 0;
    uint32_t wallclock_khz = 0;          // rate of the counter read by s_memrealtime
    uint32_t keys[SGDRC_MAX_CUS] = {};   // logical CU -> hardware key
    sgdrc_cu_mask all_cus{};
    int n_xcds = 0;
    int xcd_first_cu[kMaxXcds + 1] = {};  // logical CUs of XCD x: [first[x], first[x+1])
    // the dispatcher hands workgroup i of a grid to the XCD of workgroup
    // i mod n_xcds (checked by the topology probe); enables the static schedule
    bool static_ok = false;

    uint32_t *d_lut = nullptr;           // kLutSize entries: logical CU | group << 16
    QueueSlot *d_queues = nullptr;       // kMaxStreams
    uint64_t *d_hist_acc = nullptr;      // kMaxStreams x kHistAccCopies x kHistBins
    uint32_t *d_err = nullptr;           // one word

    void *d_scratch = nullptr;           // page-table build scratch, sized for the largest pool
    size_t scratch_bytes = 0;
    void *d_static_scratch = nullptr;    // the device address of the no-allocation build's
                                         // scratch (a static device array of colour.hip)
    uint64_t *h_pinned = nullptr;        // 8 words of pinned host memory

    uint32_t *log_cu = nullptr;
    uint32_t *log_tile = nullptr;
    uint64_t log_cap = 0;

    std::mutex mu;
    std::unordered_map<void *, StreamState> streams;
    int next_slot = 0;
    std::vector<int> free_slots;         // queue slots given back by sgdrc_stream_release
};

// A free queue slot (one released by a stream, else a new one), or -1 when
// all kMaxStreams are taken.  Caller holds c->mu.
int take_slot(Ctx *c);

// Page-table build scratch for a pool of ``pool_pages`` pages (colour.hip).
size_t pt_scratch_bytes(uint64_t pool_pages);

// Looks up the device address of the no-allocation page-table build's
// static scratch on the current device and records it in ``c`` (colour.hip;
// called by sgdrc_init with the context's device current).
int noalloc_scratch_init(Ctx *c);

// ------------------------------------------------------------ error text

int set_error(int code, const char *fmt, ...);
void clear_error();
int hip_fail(hipError_t e, const char *what);

#define SGDRC_HIP(call)                                   \
    do {                                                  \
        hipError_t e_ = (call);                           \
        if (e_ != hipSuccess)                             \
            return ::sgdrc::hip_fail(e_, #call);          \
    } while (0)

// Validates ctx and makes sure the caller's current device is ctx's.
int check_ctx(const sgdrc_ctx *ctx, Ctx **out);

// Per-stream state (creates it, with all CUs allowed, on first use).
int stream_state(Ctx *c, void *stream, StreamState **out);

// Gate arguments for a launch of ``n_tiles`` tiles on ``stream`` whose work
// queues serve runs of ``group_cus`` CUs inside an XCD (a power of two, at
// most 32), or the whole device (0).  ``preemptible``: the launch uses the
// stream's preemptible queue slot and eviction flag (the stream must have
// eviction on).
int make_gate(Ctx *c, void *stream, uint64_t n_tiles, int group_cus, Gate *g, LaunchInfo *li,
              bool preemptible = false, bool allow_static = false);

// After a launch with gate ``g`` on ``s``: if it ran the static schedule
// with a time log, enqueues the reduction of its partial end stamps into
// the log slot (k_tlog_reduce).
int finish_static_tlog(const Gate &g, hipStream_t s);

// CUs that the stream's mask allows (all CUs for a stream not seen yet).
int stream_allowed_cus(Ctx *c, void *stream);

// Whether launches on ``stream`` are to be preemptible (eviction flag set).
bool stream_preemptible(Ctx *c, void *stream);

// Enqueues, before a fresh preemptible launch on ``stream``, the discard of
// a suspended launch that was never resumed (raising
// kDevErrSuspendedDropped), so that the new launch starts on an idle slot.
int discard_suspended(Ctx *c, void *stream);

// Records ``fn`` (which has just launched with ``g``) as the stream's last
// preemptible launch, for sgdrc_resume.
void record_preemptible(Ctx *c, void *stream, const Gate &g, uint64_t n_tiles, int per_cu,
                        Relaunch fn);

// Grid size for a gated persistent kernel: the same number of workgroups
// for every CU (the dispatcher spreads them over all CUs; those on CUs
// outside the mask leave at once), as many as fit at once (or the stream's
// cap) but no more than the tiles that fall to one allowed CU.
uint32_t gated_grid(const Ctx *c, int blocks_per_cu, uint64_t n_tiles, const LaunchInfo &li);

int popcount_mask(const sgdrc_cu_mask &m);

int check_hash(const sgdrc_hash *h);
int check_shift(uint32_t page_shift);
int check_paged(const sgdrc_paged *p, const char *name);

inline Ctx *as_ctx(sgdrc_ctx *c) { return reinterpret_cast<Ctx *>(c); }

// Blocks per CU of a kernel at the given block size (cached by caller).
template <typename K>
int occupancy(K kernel, int block)
{
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, block, 0) != hipSuccess || n < 1)
        n = 1;
    return n;
}

}  // namespace sgdrc
