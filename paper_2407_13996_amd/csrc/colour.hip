// Batched XOR-hash colouring and the ordered page-table build.
//
// Colour bit k of an address is the parity of (address & M_k).  The
// classify kernel hands out tiles to single wavefronts.  A wavefront
// streams its tile's 8-byte addresses through buffer loads, each
// instruction reading 1 KiB of consecutive addresses and each lane keeping
// 8 such loads (16 addresses) in flight, colours them by table lookups
// (the hash is linear over GF(2)), and writes one colour byte per address:
// it passes its tile's 1024 colour bytes through its own 1 KiB of LDS so
// that each lane stores 16 consecutive colours per 16-byte store.  Tiles
// cover the largest multiple of 16 addresses, through buffer ranges that end
// there (so the tile body has no branch around its memory accesses); the
// last n mod 16 addresses are coloured by the grid's last workgroup.
//
// The page-table build is an ordered stream compaction over the pool's page
// addresses: a counting pass, a scan of per-workgroup counts, and an
// emitting pass that places each qualifying page with a wavefront ballot
// and a masked bit count, so the table comes out in ascending page order
// regardless of scheduling.
#include <algorithm>
#include <cstring>
#include <mutex>

#include "host_common.hpp"

namespace sgdrc {

struct HashArgs {
    uint32_t lo[SGDRC_MAX_MASKS];  // mask bits 0..31
    uint32_t hi[SGDRC_MAX_MASKS];  // mask bits 32..47
};

struct SetArgs {
    uint32_t w[8];  // 256-bit colour set
};

template <int K>
__device__ __forceinline__ uint32_t colour_of(uint32_t lo, uint32_t hi, const HashArgs &h)
{
    uint32_t c = 0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        uint32_t ones = __builtin_popcount(lo & h.lo[k]) + __builtin_popcount(hi & h.hi[k]);
        c |= (ones & 1u) << k;
    }
    return c;
}

// The hash is linear over GF(2): colour(a ^ b) = colour(a) ^ colour(b).  So
// the colour of an address is the XOR of the colours of its six bytes in
// place, colour(byte_t << 8t), each read from a 256-entry table.  A table
// is 64 LDS dwords, so a wavefront's lookups into one table conflict at most
// two ways on a bank (none with 64 banks), without replicated copies.  Six
// lookups and about ten integer ops replace the popcount form's 6 K.
constexpr int kLutBytes = 6;  // address bits 0..47

__device__ __forceinline__ uint32_t colour_lut(const uint8_t (*lut)[256], uint32_t lo, uint32_t hi)
{
    return (uint32_t)lut[0][lo & 0xffu] ^ (uint32_t)lut[1][(lo >> 8) & 0xffu] ^
           (uint32_t)lut[2][(lo >> 16) & 0xffu] ^ (uint32_t)lut[3][lo >> 24] ^
           (uint32_t)lut[4][hi & 0xffu] ^ (uint32_t)lut[5][(hi >> 8) & 0xffu];
}

// The table form of the hash (paper section 5.3): one colour byte per
// 2^shift-byte partition from ``origin``; 255 = no colour (also outside).
struct TableArgs {
    const uint8_t *lut;
    uint64_t origin;
    uint64_t entries;
    uint32_t shift;
};

__device__ __forceinline__ uint32_t table_colour(const TableArgs &t, uint64_t a)
{
    const uint64_t i = (a - t.origin) >> t.shift;
    const bool in = a >= t.origin && i < t.entries;
    return in ? (uint32_t)t.lut[in ? i : 0u] : 255u;
}

constexpr int kClsThreads = 256;
constexpr int kClsLoads = 8;                             // 16-byte loads per lane per tile
constexpr uint32_t kClsWaveTile = 64u * 2u * kClsLoads;  // 1024 addresses per wavefront
constexpr uint32_t kClsWaves = kClsThreads / 64;
// Each wavefront takes its own tiles of kClsWaveTile addresses; under a mask
// of whole XCDs by the static schedule, otherwise through work queues of 8
// CUs (one device-wide counter serialises its atomics at about 12 ns each).
constexpr int kClsGroupCus = 8;
// Two workgroups per CU with eight loads per lane: 2^26 addresses in
// 95-96 us (static) or 100 us (queues) on MI355X, against 105-125 us for one
// workgroup with 16 or 32 loads, or three with 8.
constexpr int kClsWgsPerCu = 2;
constexpr int kClsHistWgsPerCu = 2;

// Histogram bins are replicated once per lane in LDS (copy = lane), so that
// no two lanes of a wavefront ever add to one address (bin-major, so a
// wavefront's 64 adds to one bin fall in 64 consecutive dwords).  On
// MI355X, 2^26 addresses with K = 6: 97.1 us of kernel span against 99.2
// with 8, 16 or 32 copies.  16 KiB of LDS per workgroup at K = 6, 64 KiB
// for the 256 bins of a colour table (two workgroups per CU still fit).
constexpr int kHistCopies = 64;

// hist_out[b] = the sum of bin b over the kHistAccCopies accumulator copies,
// which are cleared for the next launch (every thread of one workgroup).
template <uint32_t kBins>
__device__ __forceinline__ void publish_histogram(uint64_t *hist_acc, uint64_t *hist_out)
{
    for (uint32_t b = threadIdx.x; b < kBins; b += blockDim.x) {
        uint64_t v = 0;
#pragma unroll
        for (int r = 0; r < kHistAccCopies; ++r) {
            v += __hip_atomic_load(&hist_acc[r * kHistBins + b], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&hist_acc[r * kHistBins + b], (uint64_t)0, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        hist_out[b] = v;
    }
}

// TAB: colours come from a colour table in device memory (one gathered
// byte per address) instead of the XOR hash; K is then 8 (256 bins).
template <int K, bool HIST, bool TAB>
__global__ __launch_bounds__(kClsThreads) void k_classify(const uint64_t *__restrict__ addrs,
                                                          uint64_t n, uint8_t *__restrict__ colours,
                                                          HashArgs h, TableArgs tab,
                                                          uint64_t *hist_acc, uint64_t *hist_out,
                                                          uint32_t n_tiles, Gate g)
{
    constexpr uint32_t kBins = 1u << K;
    __shared__ uint32_t s_hist[HIST ? kBins * kHistCopies : 1];
    // per wavefront: the colour bytes of one tile, 2 per lane and load
    __shared__ __attribute__((aligned(16))) uint16_t s_col[kClsThreads / 64][kClsWaveTile / 2];
    __shared__ __attribute__((aligned(16))) uint8_t s_lut[kLutBytes][256];
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t copy = lane % kHistCopies;
    const uint64_t n16 = n & ~15ull;
    if (HIST) {
        for (uint32_t i = threadIdx.x; i < kBins * kHistCopies; i += kClsThreads)
            s_hist[i] = 0;
        __syncthreads();
    }
    auto body = [&](uint32_t t, uint32_t, uint32_t &, auto &&claim) {
        // a tile is one wavefront's: its first address, and how many of its
        // addresses lie below n16 (a multiple of 16, possibly 0)
        const uint64_t base = (uint64_t)t * kClsWaveTile;
        const uint32_t valid =
            n16 > base ? (uint32_t)(n16 - base < kClsWaveTile ? n16 - base : kClsWaveTile) : 0u;
        const Rsrc ra = make_rsrc(addrs + base, valid * 8u);
        u32x4 v[kClsLoads];
#pragma unroll
        for (int j = 0; j < kClsLoads; ++j)
            v[j] = buf_load_nt(ra, (j * 64u + lane) * 16u);
        claim();
#pragma unroll
        for (int j = 0; j < kClsLoads; ++j) {
            const uint32_t c0 = TAB ? table_colour(tab, ((uint64_t)v[j].y << 32) | v[j].x)
                                    : colour_lut(s_lut, v[j].x, v[j].y);
            const uint32_t c1 = TAB ? table_colour(tab, ((uint64_t)v[j].w << 32) | v[j].z)
                                    : colour_lut(s_lut, v[j].z, v[j].w);
            s_col[wave][j * 64u + lane] = (uint16_t)(c0 | (c1 << 8));
            // both addresses of the load are valid or neither (valid is even);
            // invalid ones (read as address 0, a bin in range) add 0, so
            // that no branch splits the lanes around the atomics (with one,
            // the histogram cost several microseconds more)
            if (HIST) {
                const uint32_t inc = 2u * (j * 64u + lane) < valid ? 1u : 0u;
                atomicAdd(&s_hist[c0 * kHistCopies + copy], inc);
                atomicAdd(&s_hist[c1 * kHistCopies + copy], inc);
            }
        }
        // LDS accesses of one wavefront complete in order; the wave
        // barriers only keep the compiler from moving these accesses
        __builtin_amdgcn_wave_barrier();
        u32x4 out[kClsLoads / 8];
#pragma unroll
        for (int q = 0; q < kClsLoads / 8; ++q)
            out[q] = *reinterpret_cast<const u32x4 *>(&s_col[wave][q * 512u + lane * 8u]);
        __builtin_amdgcn_wave_barrier();
        const Rsrc rc = make_rsrc(colours + base, valid);
#pragma unroll
        for (int q = 0; q < kClsLoads / 8; ++q)
            buf_store_sc1(rc, q * 1024u + lane * 16u, out[q]);
    };
    auto flush = [&]() {
        if (HIST) {
            uint32_t xcc;
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
            uint64_t *acc = hist_acc + (xcc % (uint32_t)kHistAccCopies) * kHistBins;
            __syncthreads();
            for (uint32_t b = threadIdx.x; b < kBins; b += kClsThreads) {
                uint32_t v = 0;
#pragma unroll
                for (int r = 0; r < kHistCopies; ++r) {
                    v += s_hist[b * kHistCopies + r];
                    s_hist[b * kHistCopies + r] = 0;
                }
                if (v)
                    __hip_atomic_fetch_add(&acc[b], (uint64_t)v, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    };
    // runs in the last workgroup with every other workgroup's histogram in
    // hist_acc: colour the last n mod 16 addresses, then publish the counts
    auto epilogue = [&]() {
        const uint64_t i = n16 + threadIdx.x;
        if (i < n) {
            const uint64_t a = addrs[i];
            const uint32_t c = TAB ? table_colour(tab, a)
                                   : colour_of<K>((uint32_t)a, (uint32_t)(a >> 32), h);
            colours[i] = (uint8_t)c;
            if (HIST)
                __hip_atomic_fetch_add(&hist_acc[c], (uint64_t)1, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
        }
        if (HIST) {
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            publish_histogram<kBins>(hist_acc, hist_out);
        }
    };
    // the byte tables, visible to the whole workgroup after the loop's
    // opening barrier
    auto prologue = [&]() {
        if (TAB)
            return;
#pragma unroll
        for (int r = 0; r < kLutBytes * 256 / kClsThreads; ++r) {
            const uint32_t i = (uint32_t)r * kClsThreads + threadIdx.x;
            const uint32_t t = i >> 8, e = i & 0xffu;
            const uint64_t a = (uint64_t)e << (8u * t);
            s_lut[t][e] = (uint8_t)colour_of<K>((uint32_t)a, (uint32_t)(a >> 32), h);
        }
    };
    if (g.statics)
        static_wave_loop(g, n_tiles, prologue, body, flush);
    else
        gated_wave_loop(g, n_tiles, prologue, body, flush, epilogue);
}

// After a statically scheduled classify (one workgroup, stream-ordered
// after it): colour the last n mod 16 addresses and publish the histogram
// the workgroups accumulated in hist_acc, clearing it for the next launch.
template <int K, bool HIST, bool TAB>
__global__ __launch_bounds__(kClsThreads) void k_classify_finish(const uint64_t *__restrict__ addrs,
                                                                 uint64_t n, uint8_t *__restrict__ colours,
                                                                 HashArgs h, TableArgs tab,
                                                                 uint64_t *hist_acc, uint64_t *hist_out)
{
    constexpr uint32_t kBins = 1u << K;
    const uint64_t i = (n & ~15ull) + threadIdx.x;
    if (i < n) {
        const uint64_t a = addrs[i];
        const uint32_t c = TAB ? table_colour(tab, a) : colour_of<K>((uint32_t)a, (uint32_t)(a >> 32), h);
        colours[i] = (uint8_t)c;
        if (HIST)
            __hip_atomic_fetch_add(&hist_acc[c], (uint64_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (HIST) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        publish_histogram<kBins>(hist_acc, hist_out);
    }
}

constexpr int kPtThreads = 256;
constexpr int kPtIters = 16;
constexpr uint64_t kPtBlockPages = (uint64_t)kPtThreads * kPtIters;

// One pass of the ordered compaction.  Workgroup b covers pages
// [b*4096, (b+1)*4096) in 16 rounds of 256 consecutive pages.  The counting
// pass writes the number of qualifying pages per workgroup; the emitting
// pass writes each qualifying page at its rank among all qualifying pages.
// Page tests.  QXor: the colour of the page's base address is in the
// set given to the kernel, which the host has narrowed to the colours whose
// whole page lies in the caller's set (see page_colour_set).  QTable: every
// partition that the page touches is in the table and has a colour in the
// set.
template <int K>
struct QXor {
    HashArgs h;
    __device__ bool operator()(uint64_t a, const uint32_t *s_set) const
    {
        const uint32_t c = colour_of<K>((uint32_t)a, (uint32_t)(a >> 32), h);
        return ((s_set[c >> 5] >> (c & 31u)) & 1u) != 0u;
    }
};

struct QTable {
    TableArgs t;
    uint32_t page_shift;
    __device__ bool operator()(uint64_t a, const uint32_t *s_set) const
    {
        if (a < t.origin)
            return false;
        const uint64_t j0 = (a - t.origin) >> t.shift;
        const uint64_t j1 = (a + (1ull << page_shift) - 1u - t.origin) >> t.shift;
        if (j1 >= t.entries)
            return false;
        bool ok = true;
        for (uint64_t j = j0; j <= j1 && ok; ++j) {
            const uint32_t c = t.lut[j];
            ok = c != 255u && ((s_set[c >> 5] >> (c & 31u)) & 1u) != 0u;
        }
        return ok;
    }
};

template <class Q, bool EMIT>
__global__ __launch_bounds__(kPtThreads) void k_pt_pass(Q qual, uint64_t origin, uint32_t shift,
                                                        uint64_t pool_pages, SetArgs set,
                                                        uint32_t *block_counts,
                                                        const uint64_t *block_offsets,
                                                        uint32_t *pt, uint64_t n_needed)
{
    __shared__ uint32_t s_set[8];
    __shared__ uint32_t s_wave[kPtThreads / 64];
    if (threadIdx.x < 8)
        s_set[threadIdx.x] = set.w[threadIdx.x];
    __syncthreads();
    const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63u;
    const uint64_t base = (uint64_t)blockIdx.x * kPtBlockPages;
    uint64_t running = EMIT ? block_offsets[blockIdx.x] : 0;
    uint32_t total = 0;
    for (int it = 0; it < kPtIters; ++it) {
        const uint64_t page = base + (uint64_t)it * kPtThreads + threadIdx.x;
        const bool q = page < pool_pages && qual(origin + (page << shift), s_set);
        const uint64_t bal = __ballot(q);
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
        if (lane == 0)
            s_wave[wave] = (uint32_t)__popcll(bal);
        __syncthreads();
        uint32_t before = 0, sum = 0;
#pragma unroll
        for (uint32_t w = 0; w < kPtThreads / 64; ++w) {
            const uint32_t cw = s_wave[w];
            before += w < wave ? cw : 0u;
            sum += cw;
        }
        if (EMIT && q) {
            const uint64_t pos = running + before + below;
            if (pos < n_needed)
                pt[pos] = (uint32_t)page;
        }
        running += sum;
        total += sum;
        __syncthreads();
    }
    if (!EMIT && threadIdx.x == 0)
        block_counts[blockIdx.x] = total;
}

// Exclusive scan of the per-workgroup counts (one workgroup, chunks of 1024).
__global__ __launch_bounds__(1024) void k_pt_scan(const uint32_t *counts, uint64_t *offsets,
                                                  uint64_t nblocks, uint64_t *total)
{
    __shared__ uint64_t s[1024];
    uint64_t carry = 0;
    for (uint64_t base = 0; base < nblocks; base += 1024) {
        const uint64_t i = base + threadIdx.x;
        const uint64_t v = i < nblocks ? counts[i] : 0;
        s[threadIdx.x] = v;
        __syncthreads();
        for (uint32_t off = 1; off < 1024; off <<= 1) {
            uint64_t t = threadIdx.x >= off ? s[threadIdx.x - off] : 0;
            __syncthreads();
            s[threadIdx.x] += t;
            __syncthreads();
        }
        if (i < nblocks)
            offsets[i] = carry + s[threadIdx.x] - v;
        carry += s[1023];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        *total = carry;
}

static HashArgs hash_args(const sgdrc_hash *h)
{
    HashArgs a;
    std::memset(&a, 0, sizeof a);
    for (uint32_t k = 0; k < h->n_masks; ++k) {
        a.lo[k] = (uint32_t)h->masks[k];
        a.hi[k] = (uint32_t)(h->masks[k] >> 32);
    }
    return a;
}

template <int K, bool TAB>
static int launch_classify(Ctx *c, const HashArgs &h, const TableArgs &tab,
                           const uint64_t *d_addrs, uint64_t n, uint8_t *d_colours,
                           uint64_t *d_hist, void *stream)
{
    const uint64_t n_tiles = ((n & ~15ull) + kClsWaveTile - 1) / kClsWaveTile;
    if (n_tiles >= (1ull << 31))
        return set_error(SGDRC_EINVAL, "n too large");
    // grid sizing counts workgroups' worth of tiles
    const uint64_t wg_tiles = (n_tiles + kClsWaves - 1) / kClsWaves;
    Gate g;
    LaunchInfo li;
    int rc = make_gate(c, stream, n_tiles, kClsGroupCus, &g, &li, false, true);
    if (rc)
        return rc;
    uint64_t *acc = c->d_hist_acc + (size_t)(g.q - c->d_queues) * kHistAccCopies * kHistBins;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (d_hist) {
        static const int occ = occupancy(k_classify<K, true, TAB>, kClsThreads);
        uint32_t grid = gated_grid(c, std::min(occ, kClsHistWgsPerCu), wg_tiles, li);
        hipLaunchKernelGGL((k_classify<K, true, TAB>), dim3(grid), dim3(kClsThreads), 0, s,
                           d_addrs, n, d_colours, h, tab, acc, d_hist, (uint32_t)n_tiles, g);
    } else {
        static const int occ = occupancy(k_classify<K, false, TAB>, kClsThreads);
        uint32_t grid = gated_grid(c, std::min(occ, kClsWgsPerCu), wg_tiles, li);
        hipLaunchKernelGGL((k_classify<K, false, TAB>), dim3(grid), dim3(kClsThreads), 0, s,
                           d_addrs, n, d_colours, h, tab, acc, d_hist, (uint32_t)n_tiles, g);
    }
    SGDRC_HIP(hipGetLastError());
    if (g.statics) {
        // the statically scheduled grid has no last workgroup: the tail and
        // the histogram's publication follow in a kernel of their own
        if (d_hist)
            hipLaunchKernelGGL((k_classify_finish<K, true, TAB>), dim3(1), dim3(kClsThreads), 0, s,
                               d_addrs, n, d_colours, h, tab, acc, d_hist);
        else if (n & 15u)
            hipLaunchKernelGGL((k_classify_finish<K, false, TAB>), dim3(1), dim3(kClsThreads), 0, s,
                               d_addrs, n, d_colours, h, tab, acc, d_hist);
        SGDRC_HIP(hipGetLastError());
    }
    return finish_static_tlog(g, s);
}

template <int K>
static int launch_classify_xor(Ctx *c, const HashArgs &h, const uint64_t *d_addrs, uint64_t n,
                               uint8_t *d_colours, uint64_t *d_hist, void *stream)
{
    return launch_classify<K, false>(c, h, TableArgs{}, d_addrs, n, d_colours, d_hist, stream);
}

template <class Q>
static int launch_pagetable(Ctx *c, const Q &q, uint64_t origin, uint32_t shift,
                            uint64_t pool_pages, const SetArgs &set, uint64_t n_needed,
                            uint32_t *d_pt, uint64_t nblocks, uint32_t *d_counts,
                            uint64_t *d_offsets, uint64_t *d_total, hipStream_t s)
{
    hipLaunchKernelGGL((k_pt_pass<Q, false>), dim3((uint32_t)nblocks), dim3(kPtThreads), 0, s, q,
                       origin, shift, pool_pages, set, d_counts, (const uint64_t *)nullptr,
                       (uint32_t *)nullptr, (uint64_t)0);
    SGDRC_HIP(hipGetLastError());
    hipLaunchKernelGGL(k_pt_scan, dim3(1), dim3(1024), 0, s, (const uint32_t *)d_counts, d_offsets,
                       nblocks, d_total);
    SGDRC_HIP(hipGetLastError());
    if (n_needed > 0) {
        hipLaunchKernelGGL((k_pt_pass<Q, true>), dim3((uint32_t)nblocks), dim3(kPtThreads), 0, s,
                           q, origin, shift, pool_pages, set, d_counts,
                           (const uint64_t *)d_offsets, d_pt, n_needed);
        SGDRC_HIP(hipGetLastError());
    }
    return SGDRC_OK;
}

template <int K>
static int launch_pagetable_xor(Ctx *c, const HashArgs &h, uint64_t origin, uint32_t shift,
                                uint64_t pool_pages, const SetArgs &set, uint64_t n_needed,
                                uint32_t *d_pt, uint64_t nblocks, uint32_t *d_counts,
                                uint64_t *d_offsets, uint64_t *d_total, hipStream_t s)
{
    return launch_pagetable(c, QXor<K>{h}, origin, shift, pool_pages, set, n_needed, d_pt, nblocks,
                            d_counts, d_offsets, d_total, s);
}

// The set of base-address colours whose pages lie wholly in ``set``.  A
// page holds every address base + o, o < 2^page_shift, and the hash is
// linear over GF(2), so its bytes have exactly the colours c ^ l, with c the
// colour of its base and l running over L, the colours of the in-page
// offsets: the span of colour(1 << b) for b < page_shift.  (Paper section 6
// colours whole sectors, whose bytes share their channels.)  The page
// qualifies when that coset lies in the set.  With no mask bit below
// page_shift, L = {0} and the set is unchanged.
static sgdrc_colour_set page_colour_set(const sgdrc_hash *h, uint32_t page_shift,
                                        const sgdrc_colour_set &set)
{
    const uint32_t n = 1u << h->n_masks;
    bool in_l[256] = {};
    in_l[0] = true;
    for (uint32_t b = 0; b < page_shift && b < 48u; ++b) {
        uint32_t v = 0;
        for (uint32_t k = 0; k < h->n_masks; ++k)
            v |= (uint32_t)((h->masks[k] >> b) & 1ull) << k;
        if (in_l[v])
            continue;
        bool grown[256];
        for (uint32_t c = 0; c < n; ++c)
            grown[c] = in_l[c] || in_l[c ^ v];
        for (uint32_t c = 0; c < n; ++c)
            in_l[c] = grown[c];
    }
    auto member = [&](uint32_t c) { return ((set.bits[c >> 6] >> (c & 63u)) & 1ull) != 0ull; };
    sgdrc_colour_set out{};
    for (uint32_t c = 0; c < n; ++c) {
        bool all = true;
        for (uint32_t l = 0; l < n && all; ++l)
            all = !in_l[l] || member(c ^ l);
        if (all)
            out.bits[c >> 6] |= 1ull << (c & 63u);
    }
    return out;
}

static std::mutex g_pt_mu;  // page-table scratch is per context; builds are serialised

static int check_pool_args(uint64_t addr_origin, uint32_t page_shift, uint64_t pool_pages,
                           const sgdrc_colour_set *set, uint64_t n_needed, uint32_t *d_pt,
                           uint64_t *n_found)
{
    int rc = check_shift(page_shift);
    if (rc)
        return rc;
    if (!set || !n_found)
        return set_error(SGDRC_EINVAL, "NULL colour set or n_found");
    if (addr_origin & ((1ull << page_shift) - 1ull))
        return set_error(SGDRC_EINVAL, "addr_origin not aligned to the page size");
    if (pool_pages == 0 || pool_pages > (1ull << 32))
        return set_error(SGDRC_EINVAL, "pool_pages must be in 1..2^32");
    if (addr_origin >= (1ull << 48) || pool_pages > (((1ull << 48) - addr_origin) >> page_shift))
        return set_error(SGDRC_EINVAL, "pool extends beyond the 48-bit address space");
    if (n_needed > pool_pages)
        return set_error(SGDRC_EINVAL, "n_needed exceeds pool_pages");
    if (n_needed > 0 && (!d_pt || (reinterpret_cast<uintptr_t>(d_pt) & 3u)))
        return set_error(SGDRC_EINVAL, "page table pointer NULL or not 4-byte aligned");
    return SGDRC_OK;
}

// Every colour of the set must be below ``colours``; the set must not be empty.
static int check_set(const sgdrc_colour_set *set, uint32_t colours)
{
    bool any = false;
    for (uint32_t cc = 0; cc < 256; ++cc) {
        if ((set->bits[cc >> 6] >> (cc & 63)) & 1ull) {
            if (cc >= colours)
                return set_error(SGDRC_EINVAL, "colour %u in set, hash has %u colours", cc, colours);
            any = true;
        }
    }
    if (!any)
        return set_error(SGDRC_EINVAL, "empty colour set");
    return SGDRC_OK;
}

static int check_table(const sgdrc_colour_table *t)
{
    if (!t)
        return set_error(SGDRC_EINVAL, "colour table is NULL");
    if (t->reserved != 0)
        return set_error(SGDRC_EINVAL, "colour table reserved field must be 0");
    if (t->shift < 8 || t->shift > SGDRC_MAX_PAGE_SHIFT)
        return set_error(SGDRC_EINVAL, "partition shift %u outside [8, %d]", t->shift,
                         SGDRC_MAX_PAGE_SHIFT);
    if (t->entries > 0 && !t->lut)
        return set_error(SGDRC_EINVAL, "colour table has entries but no device pointer");
    if (t->origin >= (1ull << 48) || t->entries > (((1ull << 48) - t->origin) >> t->shift))
        return set_error(SGDRC_EINVAL, "colour table extends beyond the 48-bit address space");
    return SGDRC_OK;
}

// Scratch of one build: the scan's total (256 bytes, aligned), then the
// per-workgroup offsets (uint64) and counts (uint32).
size_t pt_scratch_bytes(uint64_t pool_pages)
{
    const uint64_t nblocks = (pool_pages + kPtBlockPages - 1) / kPtBlockPages;
    return 256 + nblocks * sizeof(uint64_t) + nblocks * sizeof(uint32_t);
}

// The no-allocation build's scratch: a fixed block of the library's own
// device memory (one per device, held until the process ends) for pools of
// up to kNoAllocMaxPages pages.  Host code never passes the array's name to
// a kernel (in host code it is only a stand-in): it uses the device address
// that noalloc_scratch_init looks up once per context, with the context's
// device current.
constexpr uint64_t kNoAllocMaxPages = 1ull << 26;
constexpr size_t kNoAllocScratch = 256 + (kNoAllocMaxPages / kPtBlockPages) * 12u;  // 192.25 KiB
static __device__ __align__(256) uint8_t scratch[kNoAllocScratch];

int noalloc_scratch_init(Ctx *c)
{
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess)
        return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p)
        return set_error(SGDRC_EHIP, "no device address for the page-table scratch");
    c->d_static_scratch = p;
    return SGDRC_OK;
}

// Enqueues the ordered compaction shared by both page tests (counting pass,
// scan, emitting pass: ``launch``) on ``s`` with the scratch at ``base``; the
// count of qualifying pages goes to *d_total.
template <class Launch>
static int enqueue_pagetable(uint64_t pool_pages, const sgdrc_colour_set *set, void *base,
                             uint64_t *d_total, hipStream_t s, Launch launch)
{
    const uint64_t nblocks = (pool_pages + kPtBlockPages - 1) / kPtBlockPages;
    uint8_t *b = static_cast<uint8_t *>(base);
    uint64_t *d_offsets = reinterpret_cast<uint64_t *>(b + 256);
    uint32_t *d_counts = reinterpret_cast<uint32_t *>(b + 256 + nblocks * sizeof(uint64_t));
    SetArgs sa;
    for (int i = 0; i < 4; ++i) {
        sa.w[2 * i] = (uint32_t)set->bits[i];
        sa.w[2 * i + 1] = (uint32_t)(set->bits[i] >> 32);
    }
    return launch(sa, nblocks, d_counts, d_offsets, d_total, s);
}

// The synchronous build: the context's scratch (allocated at init for the
// largest pool), then the count back to the host.
template <class Launch>
static int build_pagetable(Ctx *c, uint64_t pool_pages, const sgdrc_colour_set *set,
                           uint64_t n_needed, uint64_t *n_found, void *stream, Launch launch)
{
    std::lock_guard<std::mutex> lock(g_pt_mu);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (c->scratch_bytes < pt_scratch_bytes(pool_pages))
        return set_error(SGDRC_EINVAL, "pool larger than the context's page-table scratch");
    uint64_t *d_total = static_cast<uint64_t *>(c->d_scratch);
    int rc = enqueue_pagetable(pool_pages, set, c->d_scratch, d_total, s, launch);
    if (rc)
        return rc;
    SGDRC_HIP(hipMemcpyAsync(c->h_pinned, d_total, sizeof(uint64_t), hipMemcpyDeviceToHost, s));
    SGDRC_HIP(hipStreamSynchronize(s));
    *n_found = c->h_pinned[0];
    if (*n_found < n_needed)
        return set_error(SGDRC_ENOMEM, "pool holds %llu pages of the set, %llu needed",
                         (unsigned long long)*n_found, (unsigned long long)n_needed);
    return SGDRC_OK;
}

}  // namespace sgdrc

using namespace sgdrc;

#define SGDRC_DISPATCH_K(nm, fn, ...)                         \
    switch (nm) {                                             \
    case 1: rc = fn<1>(__VA_ARGS__); break;                   \
    case 2: rc = fn<2>(__VA_ARGS__); break;                   \
    case 3: rc = fn<3>(__VA_ARGS__); break;                   \
    case 4: rc = fn<4>(__VA_ARGS__); break;                   \
    case 5: rc = fn<5>(__VA_ARGS__); break;                   \
    case 6: rc = fn<6>(__VA_ARGS__); break;                   \
    case 7: rc = fn<7>(__VA_ARGS__); break;                   \
    default: rc = fn<8>(__VA_ARGS__); break;                  \
    }

extern "C" {

int colour_classify(sgdrc_ctx *ctx, const sgdrc_hash *hash, const uint64_t *d_addrs, uint64_t n,
                    uint8_t *d_colours, uint64_t *d_hist, void *stream)
{
    clear_error();
    int rc = check_hash(hash);
    if (rc)
        return rc;
    if (n > 0 && (!d_addrs || !d_colours))
        return set_error(SGDRC_EINVAL, "NULL address or colour buffer");
    if ((reinterpret_cast<uintptr_t>(d_addrs) & 15u) || (reinterpret_cast<uintptr_t>(d_colours) & 15u))
        return set_error(SGDRC_EINVAL, "address and colour buffers must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(d_hist) & 7u)
        return set_error(SGDRC_EINVAL, "histogram not 8-byte aligned");
    Ctx *c = nullptr;
    rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    HashArgs h = hash_args(hash);
    SGDRC_DISPATCH_K(hash->n_masks, launch_classify_xor, c, h, d_addrs, n, d_colours, d_hist,
                     stream);
    return rc;
}

int colour_alloc_pagetable(sgdrc_ctx *ctx, const sgdrc_hash *hash, uint64_t addr_origin,
                           uint32_t page_shift, uint64_t pool_pages, const sgdrc_colour_set *set,
                           uint64_t n_needed, uint32_t *d_pt, uint64_t *n_found, void *stream)
{
    clear_error();
    int rc = check_hash(hash);
    if (rc)
        return rc;
    if ((rc = check_pool_args(addr_origin, page_shift, pool_pages, set, n_needed, d_pt, n_found)))
        return rc;
    if ((rc = check_set(set, 1u << hash->n_masks)))
        return rc;
    Ctx *c = nullptr;
    if ((rc = check_ctx(ctx, &c)))
        return rc;
    const HashArgs h = hash_args(hash);
    const sgdrc_colour_set whole = page_colour_set(hash, page_shift, *set);
    return build_pagetable(c, pool_pages, &whole, n_needed, n_found, stream,
                           [&](const SetArgs &sa, uint64_t nblocks, uint32_t *d_counts,
                               uint64_t *d_offsets, uint64_t *d_total, hipStream_t s) {
                               int rc = SGDRC_OK;
                               SGDRC_DISPATCH_K(hash->n_masks, launch_pagetable_xor, c, h,
                                                addr_origin, page_shift, pool_pages, sa, n_needed,
                                                d_pt, nblocks, d_counts, d_offsets, d_total, s);
                               return rc;
                           });
}

int colour_alloc_pagetable_noalloc(sgdrc_ctx *ctx, const sgdrc_hash *hash, uint64_t addr_origin,
                                   uint32_t page_shift, uint64_t pool_pages,
                                   const sgdrc_colour_set *set, uint64_t n_needed, uint32_t *d_pt,
                                   uint64_t *d_n_found, void *stream)
{
    clear_error();
    int rc = check_hash(hash);
    if (rc)
        return rc;
    if ((rc = check_pool_args(addr_origin, page_shift, pool_pages, set, n_needed, d_pt,
                              d_n_found)))
        return rc;
    if (reinterpret_cast<uintptr_t>(d_n_found) & 7u)
        return set_error(SGDRC_EINVAL, "d_n_found not 8-byte aligned");
    if (pool_pages > kNoAllocMaxPages)
        return set_error(SGDRC_EINVAL, "pool_pages %llu above the %llu pages the fixed scratch "
                         "serves", (unsigned long long)pool_pages,
                         (unsigned long long)kNoAllocMaxPages);
    if ((rc = check_set(set, 1u << hash->n_masks)))
        return rc;
    Ctx *c = nullptr;
    if ((rc = check_ctx(ctx, &c)))
        return rc;
    const HashArgs h = hash_args(hash);
    const sgdrc_colour_set whole = page_colour_set(hash, page_shift, *set);
    return enqueue_pagetable(pool_pages, &whole, c->d_static_scratch, d_n_found,
                             reinterpret_cast<hipStream_t>(stream),
                             [&](const SetArgs &sa, uint64_t nblocks, uint32_t *d_counts,
                                 uint64_t *d_offsets, uint64_t *d_total, hipStream_t s) {
                                 int rc = SGDRC_OK;
                                 SGDRC_DISPATCH_K(hash->n_masks, launch_pagetable_xor, c, h,
                                                  addr_origin, page_shift, pool_pages, sa,
                                                  n_needed, d_pt, nblocks, d_counts, d_offsets,
                                                  d_total, s);
                                 return rc;
                             });
}

int colour_classify_table(sgdrc_ctx *ctx, const sgdrc_colour_table *table,
                          const uint64_t *d_addrs, uint64_t n, uint8_t *d_colours,
                          uint64_t *d_hist, void *stream)
{
    clear_error();
    int rc = check_table(table);
    if (rc)
        return rc;
    if (n > 0 && (!d_addrs || !d_colours))
        return set_error(SGDRC_EINVAL, "NULL address or colour buffer");
    if ((reinterpret_cast<uintptr_t>(d_addrs) & 15u) || (reinterpret_cast<uintptr_t>(d_colours) & 15u))
        return set_error(SGDRC_EINVAL, "address and colour buffers must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(d_hist) & 7u)
        return set_error(SGDRC_EINVAL, "histogram not 8-byte aligned");
    Ctx *c = nullptr;
    if ((rc = check_ctx(ctx, &c)))
        return rc;
    const TableArgs t{table->lut, table->origin, table->entries, table->shift};
    return launch_classify<8, true>(c, HashArgs{}, t, d_addrs, n, d_colours, d_hist, stream);
}

int colour_alloc_pagetable_table(sgdrc_ctx *ctx, const sgdrc_colour_table *table,
                                 uint64_t addr_origin, uint32_t page_shift, uint64_t pool_pages,
                                 const sgdrc_colour_set *set, uint64_t n_needed, uint32_t *d_pt,
                                 uint64_t *n_found, void *stream)
{
    clear_error();
    int rc = check_table(table);
    if (rc)
        return rc;
    if ((rc = check_pool_args(addr_origin, page_shift, pool_pages, set, n_needed, d_pt, n_found)))
        return rc;
    if ((rc = check_set(set, 255u)))
        return rc;
    Ctx *c = nullptr;
    if ((rc = check_ctx(ctx, &c)))
        return rc;
    const QTable q{TableArgs{table->lut, table->origin, table->entries, table->shift}, page_shift};
    return build_pagetable(c, pool_pages, set, n_needed, n_found, stream,
                           [&](const SetArgs &sa, uint64_t nblocks, uint32_t *d_counts,
                               uint64_t *d_offsets, uint64_t *d_total, hipStream_t s) {
                               return launch_pagetable(c, q, addr_origin, page_shift, pool_pages,
                                                       sa, n_needed, d_pt, nblocks, d_counts,
                                                       d_offsets, d_total, s);
                           });
}

}  // extern "C"
