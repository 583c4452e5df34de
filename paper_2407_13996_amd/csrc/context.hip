// Context management, CU-topology probe, per-stream CU masks and errors.
#include <algorithm>
#include <cstddef>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "host_common.hpp"

namespace sgdrc {

static thread_local std::string t_error;

int set_error(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_error = buf;
    return code;
}

void clear_error() { t_error.clear(); }

int hip_fail(hipError_t e, const char *what)
{
    return set_error(SGDRC_EHIP, "%s failed: %s", what, hipGetErrorString(e));
}

int check_ctx(const sgdrc_ctx *ctx, Ctx **out)
{
    if (!ctx)
        return set_error(SGDRC_ENODEV, "context is NULL");
    Ctx *c = reinterpret_cast<Ctx *>(const_cast<sgdrc_ctx *>(ctx));
    if (c->magic != kCtxMagic)
        return set_error(SGDRC_ENODEV, "not an initialised sgdrc context");
    int dev = -1;
    SGDRC_HIP(hipGetDevice(&dev));
    if (dev != c->device)
        return set_error(SGDRC_EINVAL, "current device %d is not the context's device %d", dev,
                         c->device);
    *out = c;
    return SGDRC_OK;
}

int popcount_mask(const sgdrc_cu_mask &m)
{
    int n = 0;
    for (int i = 0; i < 4; ++i)
        n += __builtin_popcountll(m.bits[i]);
    return n;
}

int take_slot(Ctx *c)
{
    if (!c->free_slots.empty()) {
        const int s = c->free_slots.back();
        c->free_slots.pop_back();
        return s;
    }
    return c->next_slot < kMaxStreams ? c->next_slot++ : -1;
}

int stream_state(Ctx *c, void *stream, StreamState **out)
{
    std::lock_guard<std::mutex> lock(c->mu);
    auto it = c->streams.find(stream);
    if (it == c->streams.end()) {
        const int slot = take_slot(c);
        if (slot < 0)
            return set_error(SGDRC_EINVAL, "more than %d work queues in use with one context "
                             "(sgdrc_stream_release gives a stream's back)", kMaxStreams);
        StreamState st;
        st.slot = slot;
        st.mask = c->all_cus;
        it = c->streams.emplace(stream, st).first;
    }
    *out = &it->second;
    return SGDRC_OK;
}

// Physical XCC ids whose XCD has CUs allowed by ``m``.
static uint32_t xcc_allowed(const Ctx *c, const sgdrc_cu_mask &m)
{
    uint32_t bits = 0;
    for (int x = 0; x < c->n_xcds; ++x) {
        bool any = false;
        for (int cu = c->xcd_first_cu[x]; cu < c->xcd_first_cu[x + 1] && !any; ++cu)
            any = (m.bits[cu >> 6] >> (cu & 63)) & 1ull;
        if (any)
            bits |= 1u << ((c->keys[c->xcd_first_cu[x]] >> 8) & 0xFu);
    }
    return bits;
}

int make_gate(Ctx *c, void *stream, uint64_t n_tiles, int group_cus, Gate *g, LaunchInfo *li,
              bool preemptible, bool allow_static)
{
    StreamState *st = nullptr;
    int rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    if (preemptible && st->slot_ev < 0)
        return set_error(SGDRC_EINVAL, "stream has no preemptible queue");
    std::memcpy(g->mask, st->mask.bits, sizeof g->mask);
    g->lut = c->d_lut;
    g->q = c->d_queues + (preemptible ? st->slot_ev : st->slot);
    g->evict = nullptr;
    g->resume = 0;
    if (preemptible)
        g->evict = st->evict ? st->evict
                             : reinterpret_cast<const uint32_t *>(
                                   reinterpret_cast<const char *>(g->q) + offsetof(QueueSlot, zero));
    g->evict_at = preemptible ? st->evict_at : 0u;
    g->err = c->d_err;
    g->log_cu = c->log_cu;
    g->log_tile = c->log_tile;
    g->log_cap = c->log_cap;
    g->tlog = nullptr;
    if (st->tlog) {
        g->tlog = st->tlog + 2u * (st->tlog_next % st->tlog_slots);
        ++st->tlog_next;
    }
    // queue groups: runs of group_cus CUs inside each XCD, or one group
    uint32_t shift = 0;
    while ((1 << (shift + 1)) <= group_cus && shift < 5)
        ++shift;
    const bool single = group_cus <= 0;
    if (single)
        shift = 8;  // every CU-in-XCD index (< 256) maps to sub-group 0
    uint64_t allowed[kMaxGroups] = {};
    uint64_t total = 0;
    int n_groups = 0;
    std::memset(g->grp_base, 0, sizeof g->grp_base);
    for (int x = 0; x < c->n_xcds; ++x) {
        const int first = c->xcd_first_cu[x], count = c->xcd_first_cu[x + 1] - first;
        const int subs = single ? 0 : (count + (1 << shift) - 1) >> shift;
        if (n_groups + subs > kMaxGroups)
            return set_error(SGDRC_EINVAL, "too many queue groups");
        g->grp_base[x] = (uint8_t)n_groups;
        for (int i = 0; i < count; ++i) {
            const int cu = first + i;
            const uint64_t bit = (st->mask.bits[cu >> 6] >> (cu & 63)) & 1ull;
            allowed[single ? 0 : n_groups + (i >> shift)] += bit;
            total += bit;
        }
        n_groups += subs;
    }
    if (single) {
        n_groups = 1;
        std::memset(g->grp_base, 0, sizeof g->grp_base);
    }
    uint64_t cum = 0;
    g->grp_tile[0] = 0;
    for (int grp = 0; grp < kMaxGroups; ++grp) {
        cum += allowed[grp];
        g->grp_tile[grp + 1] = (uint32_t)(total ? n_tiles * cum / total : n_tiles);
    }
    if (total == 0)
        return set_error(SGDRC_EINVAL, "the stream's CU mask allows no CU of this device");
    g->n_groups = (uint32_t)n_groups;
    g->grp_shift = shift;
    g->xcc_allowed = xcc_allowed(c, st->mask);
    // static schedule: every XCD either wholly allowed or wholly not
    g->statics = 0u;
    std::memset(g->xcd_rank, 0xFF, sizeof g->xcd_rank);
    g->n_allowed_xcd = 0u;
    g->n_xcd = (uint32_t)c->n_xcds;
    if (allow_static && !preemptible && c->static_ok) {
        bool whole = true;
        uint8_t rank[kMaxXcds];
        std::memset(rank, 0xFF, sizeof rank);
        uint32_t a = 0;
        for (int x = 0; x < c->n_xcds && whole; ++x) {
            int on = 0;
            const int first = c->xcd_first_cu[x], count = c->xcd_first_cu[x + 1] - first;
            for (int cu = first; cu < first + count; ++cu)
                on += (int)((st->mask.bits[cu >> 6] >> (cu & 63)) & 1ull);
            if (on == count)
                rank[(c->keys[first] >> 8) & 0xFu] = (uint8_t)a++;
            else if (on != 0)
                whole = false;
        }
        if (whole && a > 0) {
            g->statics = 1u;
            std::memcpy(g->xcd_rank, rank, sizeof rank);
            g->n_allowed_xcd = a;
        }
    }
    st->last_schedule = g->statics;
    st->last_tiles = n_tiles;
    li->allowed = (int)total;
    li->wg_cap = st->wg_cap;
    return SGDRC_OK;
}

// One workgroup: if the slot holds a suspended launch, drop it (zero its
// group counters and state) and raise kDevErrSuspendedDropped.  The
// arrival counters are already zero (the suspended launch reset them).
__global__ __launch_bounds__(64) void k_slot_discard(QueueSlot *q, uint32_t *err)
{
    const uint32_t st = __hip_atomic_load(&q->state[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (st != kSlotSuspended)
        return;
    __hip_atomic_store(&q->grp_next[threadIdx.x * kCounterStride], 0u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0) {
        __hip_atomic_store(&q->stopped[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&q->hb_count[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&q->hb_take[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&q->hb_limit[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&q->state[0], kSlotIdle, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        raise_flag(err, kDevErrSuspendedDropped);
    }
}

int discard_suspended(Ctx *c, void *stream)
{
    int slot;
    {
        std::lock_guard<std::mutex> lock(c->mu);
        auto it = c->streams.find(stream);
        if (it == c->streams.end() || it->second.slot_ev < 0)
            return set_error(SGDRC_EINVAL, "stream has no preemptible queue");
        slot = it->second.slot_ev;
    }
    static_assert(kMaxGroups == 64, "one thread per queue group");
    hipLaunchKernelGGL(k_slot_discard, dim3(1), dim3(64), 0, reinterpret_cast<hipStream_t>(stream),
                       c->d_queues + slot, c->d_err);
    SGDRC_HIP(hipGetLastError());
    return SGDRC_OK;
}

// One thread: store ``value`` to the flag and stamp the device wall clock.
__global__ __launch_bounds__(64) void k_signal_flag(uint32_t *flag, uint32_t value, uint64_t *stamp)
{
    if (threadIdx.x != 0)
        return;
    __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (stamp)
        __hip_atomic_store(stamp, __builtin_amdgcn_s_memrealtime(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// One wavefront: the end stamp of a statically scheduled launch is the
// largest of its partial end stamps, which are cleared for the next launch.
__global__ __launch_bounds__(64) void k_tlog_reduce(QueueSlot *q, uint64_t *tlog)
{
    uint64_t *p = &q->tpart[threadIdx.x * (kCounterStride / 2)];
    uint64_t v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(p, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint64_t o = __shfl_xor(v, off, 64);
        v = o > v ? o : v;
    }
    if (threadIdx.x == 0)
        __hip_atomic_store(&tlog[1], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

int finish_static_tlog(const Gate &g, hipStream_t s)
{
    if (!g.statics || !g.tlog)
        return SGDRC_OK;
    static_assert(kTimePartials == 64, "one lane per partial");
    hipLaunchKernelGGL(k_tlog_reduce, dim3(1), dim3(64), 0, s, g.q, g.tlog);
    SGDRC_HIP(hipGetLastError());
    return SGDRC_OK;
}

int stream_allowed_cus(Ctx *c, void *stream)
{
    std::lock_guard<std::mutex> lock(c->mu);
    auto it = c->streams.find(stream);
    return popcount_mask(it != c->streams.end() ? it->second.mask : c->all_cus);
}

bool stream_preemptible(Ctx *c, void *stream)
{
    std::lock_guard<std::mutex> lock(c->mu);
    auto it = c->streams.find(stream);
    return it != c->streams.end() && it->second.ev_on;
}

void record_preemptible(Ctx *c, void *stream, const Gate &g, uint64_t n_tiles, int per_cu,
                        Relaunch fn)
{
    std::lock_guard<std::mutex> lock(c->mu);
    StreamState &st = c->streams[stream];
    st.ev_gate = g;
    st.ev_tiles = n_tiles;
    st.ev_per_cu = per_cu;
    st.ev_relaunch = std::move(fn);
}

uint32_t gated_grid(const Ctx *c, int blocks_per_cu, uint64_t n_tiles, const LaunchInfo &li)
{
    uint64_t fit = (uint64_t)blocks_per_cu;
    if (li.wg_cap)
        fit = std::min<uint64_t>(fit, li.wg_cap);
    const uint64_t allowed = (uint64_t)std::max(li.allowed, 1);
    const uint64_t per_cu_tiles = (n_tiles + allowed - 1) / allowed;
    const uint64_t per_cu = std::max<uint64_t>(1, std::min<uint64_t>(fit, per_cu_tiles));
    return (uint32_t)(per_cu * (uint64_t)c->num_cus);
}

int check_hash(const sgdrc_hash *h)
{
    if (!h)
        return set_error(SGDRC_EINVAL, "hash is NULL");
    if (h->n_masks < 1 || h->n_masks > SGDRC_MAX_MASKS)
        return set_error(SGDRC_EINVAL, "n_masks %u outside 1..%d", h->n_masks, SGDRC_MAX_MASKS);
    if (h->reserved != 0)
        return set_error(SGDRC_EINVAL, "hash.reserved must be 0");
    for (uint32_t k = 0; k < h->n_masks; ++k)
        if (h->masks[k] >> 48)
            return set_error(SGDRC_EINVAL, "mask %u selects address bits above 47", k);
    return SGDRC_OK;
}

int check_shift(uint32_t page_shift)
{
    if (page_shift < SGDRC_MIN_PAGE_SHIFT || page_shift > SGDRC_MAX_PAGE_SHIFT)
        return set_error(SGDRC_EINVAL, "page_shift %u outside [%d, %d]", page_shift,
                         SGDRC_MIN_PAGE_SHIFT, SGDRC_MAX_PAGE_SHIFT);
    return SGDRC_OK;
}

int check_paged(const sgdrc_paged *p, const char *name)
{
    if (!p)
        return set_error(SGDRC_EINVAL, "%s is NULL", name);
    if (!p->pool || !p->pt)
        return set_error(SGDRC_EINVAL, "%s: NULL pool or page table", name);
    if (reinterpret_cast<uintptr_t>(p->pool) & 255u)
        return set_error(SGDRC_EINVAL, "%s: pool not 256-byte aligned", name);
    if (reinterpret_cast<uintptr_t>(p->pt) & 3u)
        return set_error(SGDRC_EINVAL, "%s: page table not 4-byte aligned", name);
    if (p->pool_pages == 0)
        return set_error(SGDRC_EINVAL, "%s: pool_pages is 0", name);
    return SGDRC_OK;
}

// Each workgroup records the hardware key of the CU it runs on; the sleep
// keeps workgroups resident long enough for the dispatcher to spread the
// grid over every CU.
__global__ void k_cu_probe(uint32_t *keys, uint32_t n, uint32_t spins)
{
    uint32_t key = hw_key();
    for (uint32_t i = 0; i < spins; ++i)
        __builtin_amdgcn_s_sleep(8);
    if (threadIdx.x == 0 && blockIdx.x < n)
        keys[blockIdx.x] = key;
}

// Whether workgroup i of the probe grid ran on the XCD of workgroup
// i mod n_xcds, with the first n_xcds workgroups on n_xcds different XCDs
// (the partition the static schedule relies on).
static bool xcd_partition_holds(const std::vector<uint32_t> &raw, int n_xcds)
{
    if (n_xcds < 1 || raw.size() < (size_t)n_xcds || raw.size() % (size_t)n_xcds)
        return false;
    uint32_t seen = 0;
    for (int r = 0; r < n_xcds; ++r)
        seen |= 1u << ((raw[r] >> 8) & 0xFu);
    if (__builtin_popcount(seen) != n_xcds)
        return false;
    for (size_t i = 0; i < raw.size(); ++i)
        if (((raw[i] ^ raw[i % n_xcds]) >> 8) & 0xFu)
            return false;
    return true;
}

static int probe_topology(Ctx *c, int expected)
{
    std::vector<uint32_t> uniq, raw;
    for (int attempt = 0; attempt < 3; ++attempt) {
        const uint32_t n = (uint32_t)expected * (48u << attempt);
        uint32_t *d_keys = nullptr;
        SGDRC_HIP(hipMalloc(&d_keys, n * sizeof(uint32_t)));
        hipLaunchKernelGGL(k_cu_probe, dim3(n), dim3(64), 0, 0, d_keys, n, 32u << attempt);
        hipError_t e = hipGetLastError();
        if (e == hipSuccess)
            e = hipDeviceSynchronize();
        std::vector<uint32_t> keys(n);
        if (e == hipSuccess)
            e = hipMemcpy(keys.data(), d_keys, n * sizeof(uint32_t), hipMemcpyDeviceToHost);
        (void)hipFree(d_keys);
        if (e != hipSuccess)
            return hip_fail(e, "CU probe");
        raw = keys;
        std::sort(keys.begin(), keys.end());
        keys.erase(std::unique(keys.begin(), keys.end()), keys.end());
        uniq = keys;
        if ((int)uniq.size() >= expected)
            break;
    }
    if ((int)uniq.size() != expected)
        return set_error(SGDRC_ENODEV, "CU probe found %zu distinct CUs, device reports %d",
                         uniq.size(), expected);
    if (expected > SGDRC_MAX_CUS)
        return set_error(SGDRC_ENODEV, "device has %d CUs, more than %d", expected,
                         SGDRC_MAX_CUS);
    // XCDs: CUs with the same XCC_ID (key bits 11:8), in key order
    std::vector<uint32_t> lut(kLutSize, kLutNone);
    int n_xcds = 0;
    for (int i = 0; i < expected; ++i) {
        if (uniq[i] >= (uint32_t)kLutSize)
            return set_error(SGDRC_ENODEV, "CU key 0x%x out of range", uniq[i]);
        if (i == 0 || (uniq[i] >> 8) != (uniq[i - 1] >> 8)) {
            if (n_xcds == kMaxXcds)
                return set_error(SGDRC_ENODEV, "more than %d XCCs", kMaxXcds);
            c->xcd_first_cu[n_xcds++] = i;
        }
        const uint32_t in_xcd = (uint32_t)(i - c->xcd_first_cu[n_xcds - 1]);
        if (in_xcd > 255u)
            return set_error(SGDRC_ENODEV, "more than 256 CUs in one XCC");
        c->keys[i] = uniq[i];
        lut[uniq[i]] = (uint32_t)i | ((uint32_t)(n_xcds - 1) << 16) | (in_xcd << 24);
    }
    c->n_xcds = n_xcds;
    for (int x = n_xcds; x <= kMaxXcds; ++x)
        c->xcd_first_cu[x] = expected;
    c->static_ok = xcd_partition_holds(raw, n_xcds);
    c->num_cus = expected;
    std::memset(&c->all_cus, 0, sizeof c->all_cus);
    for (int i = 0; i < expected; ++i)
        c->all_cus.bits[i >> 6] |= 1ull << (i & 63);
    SGDRC_HIP(hipMemcpy(c->d_lut, lut.data(), kLutSize * sizeof(uint32_t), hipMemcpyHostToDevice));
    return SGDRC_OK;
}

static void free_ctx(Ctx *c)
{
    if (c->d_lut) (void)hipFree(c->d_lut);
    if (c->d_queues) (void)hipFree(c->d_queues);
    if (c->d_hist_acc) (void)hipFree(c->d_hist_acc);
    if (c->d_err) (void)hipFree(c->d_err);
    if (c->d_scratch) (void)hipFree(c->d_scratch);
    if (c->h_pinned) (void)hipHostFree(c->h_pinned);
    c->magic = 0;
    delete c;
}

}  // namespace sgdrc

using namespace sgdrc;

extern "C" {

int sgdrc_init(int device, sgdrc_ctx **out)
{
    clear_error();
    if (!out)
        return set_error(SGDRC_EINVAL, "out is NULL");
    *out = nullptr;
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || count <= 0)
        return set_error(SGDRC_ENODEV, "no HIP device");
    if (device < 0 || device >= count)
        return set_error(SGDRC_ENODEV, "device %d outside 0..%d", device, count - 1);
    hipDeviceProp_t prop;
    SGDRC_HIP(hipGetDeviceProperties(&prop, device));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return set_error(SGDRC_ENODEV, "device %d is %s, not gfx950", device, prop.gcnArchName);
    SGDRC_HIP(hipSetDevice(device));

    Ctx *c = new (std::nothrow) Ctx();
    if (!c)
        return set_error(SGDRC_EHIP, "out of host memory");
    c->device = device;
    {
        int khz = 0;
        SGDRC_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, device));
        c->wallclock_khz = khz > 0 ? (uint32_t)khz : 0u;
    }
    int rc = SGDRC_OK;
    hipError_t e = hipSuccess;
#define TRY(call)                                   \
    do {                                            \
        e = (call);                                 \
        if (e != hipSuccess) {                      \
            rc = hip_fail(e, #call);                \
            free_ctx(c);                            \
            return rc;                              \
        }                                           \
    } while (0)
    TRY(hipMalloc(&c->d_lut, kLutSize * sizeof(uint32_t)));
    TRY(hipMalloc(&c->d_queues, kMaxStreams * sizeof(QueueSlot)));
    TRY(hipMemset(c->d_queues, 0, kMaxStreams * sizeof(QueueSlot)));
    TRY(hipMalloc(&c->d_hist_acc,
                  (size_t)kMaxStreams * kHistAccCopies * kHistBins * sizeof(uint64_t)));
    TRY(hipMemset(c->d_hist_acc, 0,
                  (size_t)kMaxStreams * kHistAccCopies * kHistBins * sizeof(uint64_t)));
    TRY(hipMalloc(&c->d_err, sizeof(uint32_t)));
    TRY(hipMemset(c->d_err, 0, sizeof(uint32_t)));
    TRY(hipHostMalloc(&c->h_pinned, 8 * sizeof(uint64_t), hipHostMallocDefault));
    // the page-table build's scratch for the largest pool (2^32 pages): a
    // build never allocates, so it never waits for the whole device
    c->scratch_bytes = pt_scratch_bytes(1ull << 32);
    TRY(hipMalloc(&c->d_scratch, c->scratch_bytes));
#undef TRY
    rc = noalloc_scratch_init(c);
    if (rc) {
        free_ctx(c);
        return rc;
    }
    rc = probe_topology(c, prop.multiProcessorCount);
    if (rc) {
        free_ctx(c);
        return rc;
    }
    *out = reinterpret_cast<sgdrc_ctx *>(c);
    return SGDRC_OK;
}

int sgdrc_destroy(sgdrc_ctx *ctx)
{
    clear_error();
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    SGDRC_HIP(hipDeviceSynchronize());
    free_ctx(c);
    return SGDRC_OK;
}

int sgdrc_num_cus(const sgdrc_ctx *ctx)
{
    if (!ctx)
        return set_error(SGDRC_ENODEV, "context is NULL");
    const Ctx *c = reinterpret_cast<const Ctx *>(ctx);
    if (c->magic != kCtxMagic)
        return set_error(SGDRC_ENODEV, "not an initialised sgdrc context");
    return c->num_cus;
}

int sgdrc_cu_key(const sgdrc_ctx *ctx, uint32_t cu, uint32_t *key)
{
    if (!key)
        return set_error(SGDRC_EINVAL, "key is NULL");
    int n = sgdrc_num_cus(ctx);
    if (n < 0)
        return n;
    if (cu >= (uint32_t)n)
        return set_error(SGDRC_EINVAL, "cu %u >= %d", cu, n);
    *key = reinterpret_cast<const Ctx *>(ctx)->keys[cu];
    return SGDRC_OK;
}

const char *sgdrc_last_error(void) { return t_error.c_str(); }

int sgdrc_device_error(sgdrc_ctx *ctx, uint32_t *flags)
{
    clear_error();
    if (!flags)
        return set_error(SGDRC_EINVAL, "flags is NULL");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    SGDRC_HIP(hipDeviceSynchronize());
    SGDRC_HIP(hipMemcpy(flags, c->d_err, sizeof(uint32_t), hipMemcpyDeviceToHost));
    SGDRC_HIP(hipMemset(c->d_err, 0, sizeof(uint32_t)));
    SGDRC_HIP(hipDeviceSynchronize());
    return SGDRC_OK;
}

int sgdrc_set_worklog(sgdrc_ctx *ctx, uint32_t *d_cu_tiles, uint32_t *d_tile_visits,
                      uint64_t tile_cap)
{
    clear_error();
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    c->log_cu = d_cu_tiles;
    c->log_tile = d_tile_visits;
    c->log_cap = d_tile_visits ? tile_cap : 0;
    return SGDRC_OK;
}

int sgdrc_last_tiles(sgdrc_ctx *ctx, void *stream, uint64_t *tiles)
{
    clear_error();
    if (!tiles)
        return set_error(SGDRC_EINVAL, "tiles is NULL");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    auto it = c->streams.find(stream);
    *tiles = it == c->streams.end() ? 0 : it->second.last_tiles;
    return SGDRC_OK;
}

int sgdrc_last_schedule(sgdrc_ctx *ctx, void *stream, uint32_t *schedule)
{
    clear_error();
    if (!schedule)
        return set_error(SGDRC_EINVAL, "schedule is NULL");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    auto it = c->streams.find(stream);
    *schedule = it == c->streams.end() ? 0u : it->second.last_schedule;
    return SGDRC_OK;
}

int sgdrc_set_timelog(sgdrc_ctx *ctx, void *stream, uint64_t *d_slots, uint32_t n_slots)
{
    clear_error();
    if (d_slots && n_slots == 0)
        return set_error(SGDRC_EINVAL, "n_slots is 0");
    if (reinterpret_cast<uintptr_t>(d_slots) & 7u)
        return set_error(SGDRC_EINVAL, "time-log slots not 8-byte aligned");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    st->tlog = d_slots;
    st->tlog_slots = d_slots ? n_slots : 0;
    st->tlog_next = 0;
    return SGDRC_OK;
}

int sgdrc_wallclock_khz(const sgdrc_ctx *ctx, uint32_t *khz)
{
    clear_error();
    if (!khz)
        return set_error(SGDRC_EINVAL, "khz is NULL");
    Ctx *c = nullptr;
    int rc = check_ctx(const_cast<sgdrc_ctx *>(ctx), &c);
    if (rc)
        return rc;
    *khz = c->wallclock_khz;
    return SGDRC_OK;
}

int sgdrc_set_stream_occupancy(sgdrc_ctx *ctx, void *stream, uint32_t max_wgs_per_cu)
{
    clear_error();
    if (max_wgs_per_cu > 64)
        return set_error(SGDRC_EINVAL, "max_wgs_per_cu %u above 64", max_wgs_per_cu);
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    st->wg_cap = max_wgs_per_cu;
    return SGDRC_OK;
}

int set_cu_mask(sgdrc_ctx *ctx, void *stream, const sgdrc_cu_mask *mask)
{
    clear_error();
    if (mask && popcount_mask(*mask) == 0)
        return set_error(SGDRC_EINVAL, "empty CU mask");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    if (mask) {
        for (int i = c->num_cus; i < SGDRC_MAX_CUS; ++i)
            if ((mask->bits[i >> 6] >> (i & 63)) & 1ull)
                return set_error(SGDRC_EINVAL, "CU mask names CU %d, device has %d", i,
                                 c->num_cus);
    }
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    st->mask = mask ? *mask : c->all_cus;
    return SGDRC_OK;
}

int sgdrc_set_eviction_flag(sgdrc_ctx *ctx, void *stream, const uint32_t *d_flag)
{
    clear_error();
    if (reinterpret_cast<uintptr_t>(d_flag) & 3u)
        return set_error(SGDRC_EINVAL, "eviction flag not 4-byte aligned");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    if (d_flag && st->slot_ev < 0) {
        const int slot = take_slot(c);
        if (slot < 0)
            return set_error(SGDRC_EINVAL, "more than %d work queues in use with one context "
                             "(sgdrc_stream_release gives a stream's back)", kMaxStreams);
        st->slot_ev = slot;
    }
    st->ev_on = d_flag != nullptr;
    st->evict = d_flag;
    return SGDRC_OK;
}

int sgdrc_set_eviction_hook(sgdrc_ctx *ctx, void *stream, uint32_t tile)
{
    clear_error();
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(c->mu);
    st->evict_at = tile;
    return SGDRC_OK;
}

int sgdrc_stream_release(sgdrc_ctx *ctx, void *stream)
{
    clear_error();
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    int slot = -1, slot_ev = -1;
    {
        std::lock_guard<std::mutex> lock(c->mu);
        auto it = c->streams.find(stream);
        if (it == c->streams.end())
            return SGDRC_OK;
        slot = it->second.slot;
        slot_ev = it->second.slot_ev;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    SGDRC_HIP(hipStreamSynchronize(s));
    if (slot_ev >= 0) {
        // a suspended launch that was never resumed is dropped, so that the
        // slot is idle for its next owner
        hipLaunchKernelGGL(k_slot_discard, dim3(1), dim3(64), 0, s, c->d_queues + slot_ev,
                           c->d_err);
        SGDRC_HIP(hipGetLastError());
        SGDRC_HIP(hipStreamSynchronize(s));
    }
    std::lock_guard<std::mutex> lock(c->mu);
    c->streams.erase(stream);
    if (slot >= 0)
        c->free_slots.push_back(slot);
    if (slot_ev >= 0)
        c->free_slots.push_back(slot_ev);
    return SGDRC_OK;
}

int sgdrc_resume(sgdrc_ctx *ctx, void *stream)
{
    clear_error();
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    Relaunch fn;
    Gate g;
    LaunchInfo li;
    uint64_t tiles = 0;
    int per_cu = 1;
    {
        std::lock_guard<std::mutex> lock(c->mu);
        if (!st->ev_relaunch)
            return set_error(SGDRC_EINVAL, "no preemptible launch on this stream to resume");
        const int allowed = popcount_mask(st->mask);
        if (allowed == 0)
            return set_error(SGDRC_EINVAL, "the stream's CU mask allows no CU of this device");
        // the suspended launch's tile ranges and group layout, the current
        // mask, flag and logs
        g = st->ev_gate;
        std::memcpy(g.mask, st->mask.bits, sizeof g.mask);
        g.xcc_allowed = xcc_allowed(c, st->mask);
        g.q = c->d_queues + st->slot_ev;
        g.evict = st->evict ? st->evict
                            : reinterpret_cast<const uint32_t *>(
                                  reinterpret_cast<const char *>(g.q) + offsetof(QueueSlot, zero));
        g.resume = 1;
        g.evict_at = st->evict_at;
        g.log_cu = c->log_cu;
        g.log_tile = c->log_tile;
        g.log_cap = c->log_cap;
        g.tlog = nullptr;
        if (st->tlog) {
            g.tlog = st->tlog + 2u * (st->tlog_next % st->tlog_slots);
            ++st->tlog_next;
        }
        tiles = st->ev_tiles;
        per_cu = st->ev_per_cu;
        st->last_tiles = tiles;
        li.allowed = allowed;
        li.wg_cap = st->wg_cap;
        fn = st->ev_relaunch;
    }
    SGDRC_HIP(fn(g, gated_grid(c, per_cu, tiles, li)));
    return SGDRC_OK;
}

int sgdrc_suspended(sgdrc_ctx *ctx, void *stream, uint64_t *tiles_left)
{
    clear_error();
    if (!tiles_left)
        return set_error(SGDRC_EINVAL, "tiles_left is NULL");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    StreamState *st = nullptr;
    rc = stream_state(c, stream, &st);
    if (rc)
        return rc;
    int slot;
    Gate g;
    {
        std::lock_guard<std::mutex> lock(c->mu);
        if (!st->ev_relaunch)
            return set_error(SGDRC_EINVAL, "no preemptible launch on this stream");
        slot = st->slot_ev;
        g = st->ev_gate;
    }
    SGDRC_HIP(hipStreamSynchronize(reinterpret_cast<hipStream_t>(stream)));
    QueueSlot q;
    SGDRC_HIP(hipMemcpy(&q, c->d_queues + slot, sizeof q, hipMemcpyDeviceToHost));
    uint64_t left = 0;
    if (q.state[0] == kSlotSuspended) {
        for (uint32_t i = 0; i < g.n_groups; ++i) {
            const uint32_t size = g.grp_tile[i + 1] - g.grp_tile[i];
            const uint32_t taken = q.grp_next[i * kCounterStride];
            left += taken < size ? size - taken : 0u;
        }
        // tiles handed back by stopped workgroups (the suspension set the
        // ring's claim counter to the first of them)
        left += q.hb_count[0] - q.hb_take[0];
    }
    *tiles_left = left;
    return SGDRC_OK;
}

int sgdrc_tidal_masks(uint32_t num_cus, const uint32_t *ls_cus, uint32_t n_queued,
                      uint32_t window, uint32_t granule, sgdrc_cu_mask *ls_mask,
                      sgdrc_cu_mask *be_mask)
{
    clear_error();
    if (num_cus < 1 || num_cus > SGDRC_MAX_CUS)
        return set_error(SGDRC_EINVAL, "num_cus %u outside 1..%d", num_cus, SGDRC_MAX_CUS);
    if (window < 1 || granule < 1)
        return set_error(SGDRC_EINVAL, "window and granule must be positive");
    if (n_queued > 0 && !ls_cus)
        return set_error(SGDRC_EINVAL, "ls_cus is NULL");
    if (!ls_mask || !be_mask)
        return set_error(SGDRC_EINVAL, "NULL mask");
    uint32_t need = 0;
    for (uint32_t i = 0; i < n_queued && i < window; ++i) {
        if (ls_cus[i] > num_cus)
            return set_error(SGDRC_EINVAL, "queued kernel %u needs %u CUs, device has %u", i,
                             ls_cus[i], num_cus);
        need = std::max(need, ls_cus[i]);
    }
    uint64_t r = ((uint64_t)need + granule - 1) / granule * granule;
    if (r > num_cus)
        r = num_cus;
    std::memset(ls_mask, 0, sizeof *ls_mask);
    std::memset(be_mask, 0, sizeof *be_mask);
    for (uint32_t cu = 0; cu < num_cus; ++cu) {
        sgdrc_cu_mask *m = cu < r ? ls_mask : be_mask;
        m->bits[cu >> 6] |= 1ull << (cu & 63);
    }
    return SGDRC_OK;
}

int sgdrc_signal_flag(sgdrc_ctx *ctx, void *stream, uint32_t *d_flag, uint32_t value,
                      uint64_t *d_stamp)
{
    clear_error();
    if (!d_flag || (reinterpret_cast<uintptr_t>(d_flag) & 3u))
        return set_error(SGDRC_EINVAL, "flag NULL or not 4-byte aligned");
    if (reinterpret_cast<uintptr_t>(d_stamp) & 7u)
        return set_error(SGDRC_EINVAL, "stamp not 8-byte aligned");
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    hipLaunchKernelGGL(k_signal_flag, dim3(1), dim3(64), 0, reinterpret_cast<hipStream_t>(stream),
                       d_flag, value, d_stamp);
    SGDRC_HIP(hipGetLastError());
    return SGDRC_OK;
}

}  // extern "C"
