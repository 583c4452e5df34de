// Page-table-indirected streaming kernels: bimodal relayout (page-set to
// page-set copy) and the colour-restricted triad a = b + s*c.
//
// Both run as gated persistent grids over a tile queue, one workgroup per
// CU.  A tile is 64 KiB of logical bytes per array; each of the four
// wavefronts of a workgroup owns 16 KiB of it, and every lane moves 16
// chunks of 16 bytes (256 bytes in flight per lane and array) with
// non-temporal buffer loads and stores, each wavefront instruction covering
// 1 KiB of consecutive bytes.
//
// The tile's page-table entries (one to sixteen pages) are staged in LDS.
// Every 1 KiB wavefront chunk lies inside one page, and each gets its own
// buffer resource: base = the chunk's address in its page, range = the
// bytes the chunk may touch (zero for an out-of-range page-table entry,
// fewer for the last tile).  The hardware drops accesses outside the range,
// so the tile body is the same straight-line code for full, ragged and
// skipped chunks.  That matters for speed as well as brevity: the next
// tile's ticket is requested between the loads and the stores, and its
// result is waited for only after the stores have been issued; a branch in
// the body would make the compiler wait for the stores too on the way to
// the next tile.  (One resource per chunk also measured faster than one
// resource per tile and array with offsets up to 64 KiB: 6.5-6.7 against
// 5.9-6.5 TB/s for the triad on 64 KiB pages.)
//
// Tiles cover the largest multiple of 16 bytes; the last n_bytes mod 16
// bytes are moved by the last workgroup of the grid after all tiles are
// done (it may sit on any CU).
#include "host_common.hpp"

namespace sgdrc {

constexpr int kStreamThreads = 256;
constexpr uint32_t kStepSpan = 64u * 16u;  // 1 KiB per wavefront instruction

// Tile geometry for U 16-byte chunks per lane and array.
template <int U>
struct Geo {
    static constexpr uint32_t kTile = (uint32_t)kStreamThreads * 16u * U;
    static constexpr uint32_t kWaveSpan = 64u * 16u * U;
    static constexpr int kPagesMax = (int)(kTile >> SGDRC_MIN_PAGE_SHIFT);
};

// Chunks per lane and array (tile = 4 KiB x U) and workgroups per CU.
// Few deep workgroups measured fastest on MI355X: one 256-thread workgroup
// per CU (one wavefront per SIMD) with 16 loads of 16 bytes per lane and
// array in flight moves 1 GiB arrays at 6.4-6.7 TB/s, for the triad and for
// the copy alike; a second workgroup per CU, or 8 loads per lane, costs 5
// to 20 percent.
constexpr int kTriadUnroll = 16;
// Preemptible triad launches: a workgroup stops after the tile it is on and
// the one it has already claimed, so the tile size bounds the eviction delay.
constexpr int kTriadUnrollEv = 16;
constexpr int kRelayoutUnroll = 16;
constexpr int kStreamWgsPerCu = 1;
// each workgroup of a preemptible launch hands back at most one tile
static_assert(2 * kStreamWgsPerCu * kMaxCus <= (int)kHandBackCap, "hand-back ring too small");

// Bytes of the span [from, from + span) that lie below n16.
__device__ __forceinline__ uint32_t span_valid(uint64_t from, uint64_t n16, uint32_t span)
{
    return n16 > from ? (uint32_t)(n16 - from < span ? n16 - from : span) : 0u;
}

// Wavefront index, known to the compiler to be uniform.
__device__ __forceinline__ uint32_t wave_id()
{
    return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

// Resource for the 1 KiB chunk at logical byte ``at`` (inside pool page p;
// kBadPage gives an empty range).
__device__ __forceinline__ Rsrc chunk_rsrc(const uint8_t *pool, uint32_t p, uint32_t shift,
                                           uint64_t pmask, uint64_t at, uint32_t valid)
{
    const bool ok = p != kBadPage;
    return make_rsrc(pool + (ok ? ((uint64_t)p << shift) + (at & pmask) : 0u), ok ? valid : 0u);
}

// Stages the entries of the pages that tile [t0, t0 + tile) touches: entry
// i of each table is for logical page (t0 >> shift) + i.  Pages at or beyond
// n_pages, and entries out of range of their pool, become kBadPage (the
// latter also set the error bit).  ALL3: a page is kept only if it is valid
// in every table.
template <int N, bool ALL3>
__device__ __forceinline__ void stage_tile_pages(uint64_t t0, uint32_t tile, uint32_t shift,
                                                 uint64_t n_pages, const uint32_t *const pts[N],
                                                 const uint64_t pool_pages[N], uint32_t *const s[N],
                                                 uint32_t &err)
{
    const uint64_t p0 = t0 >> shift;
    const uint32_t np = (uint32_t)(((t0 + tile - 1u) >> shift) - p0 + 1u);
    if (threadIdx.x < np) {
        const uint64_t j = p0 + threadIdx.x;
        uint32_t p[N];
        bool ok = true;
#pragma unroll
        for (int a = 0; a < N; ++a) {
            p[a] = j < n_pages ? checked_page(pts[a], j, pool_pages[a], err) : kBadPage;
            ok = ok && p[a] != kBadPage;
        }
#pragma unroll
        for (int a = 0; a < N; ++a)
            s[a][threadIdx.x] = (ALL3 && !ok) ? kBadPage : p[a];
    }
    __syncthreads();
}

// One relayout tile (tile t of a copy of n_bytes logical bytes) for the
// batched kernel: stage the tile's entries of both tables, load each
// wavefront chunk from its source page, claim the next ticket, store each
// chunk to its destination page.  (k_relayout below keeps the same steps
// written out in its own body: sharing this function cost the single-copy
// kernel 0.6 percent on MI355X.)
template <int U, typename Claim_>
__device__ __forceinline__ void relayout_tile(uint8_t *dst, const uint32_t *pt_d, uint64_t dst_pages,
                                              const uint8_t *src, const uint32_t *pt_s,
                                              uint64_t src_pages, uint64_t n_bytes, uint32_t shift,
                                              uint32_t t, uint32_t *s_pd, uint32_t *s_ps,
                                              uint32_t &err, Claim_ &&claim)
{
    constexpr uint32_t kTile = Geo<U>::kTile;
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t n16 = n_bytes & ~15ull;
    const uint64_t n_pages = (n16 + pmask) >> shift;
    const uint32_t lane16 = (threadIdx.x & 63u) * 16u;
    const uint32_t wbase = wave_id() * Geo<U>::kWaveSpan;
    const uint32_t *const pts[2] = {pt_d, pt_s};
    const uint64_t pools[2] = {dst_pages, src_pages};
    uint32_t *const stg[2] = {s_pd, s_ps};
    const uint64_t t0 = (uint64_t)t * kTile;
    const uint64_t p0 = t0 >> shift;
    stage_tile_pages<2, true>(t0, kTile, shift, n_pages, pts, pools, stg, err);
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint64_t at = t0 + wbase + u * kStepSpan;
        const uint32_t jl = (uint32_t)((at >> shift) - p0);
        const uint32_t ps = __builtin_amdgcn_readfirstlane(s_ps[jl]);
        v[u] = buf_load_nt(chunk_rsrc(src, ps, shift, pmask, at, span_valid(at, n16, kStepSpan)),
                           lane16);
    }
    claim();
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint64_t at = t0 + wbase + u * kStepSpan;
        const uint32_t jl = (uint32_t)((at >> shift) - p0);
        const uint32_t pd = __builtin_amdgcn_readfirstlane(s_pd[jl]);
        buf_store_nt(chunk_rsrc(dst, pd, shift, pmask, at, span_valid(at, n16, kStepSpan)),
                     lane16, v[u]);
    }
    __syncthreads();
}

// The last n_bytes mod 16 bytes of a copy, all inside the page that holds
// byte n_bytes & ~15 (threads 0..14).
__device__ __forceinline__ void relayout_tail(uint8_t *dst, const uint32_t *pt_d, uint64_t dst_pages,
                                              const uint8_t *src, const uint32_t *pt_s,
                                              uint64_t src_pages, uint64_t n_bytes, uint32_t shift,
                                              uint32_t *err_word)
{
    const uint64_t n16 = n_bytes & ~15ull;
    const uint32_t rem = (uint32_t)(n_bytes - n16);
    if (threadIdx.x < rem) {
        const uint64_t pmask = (1ull << shift) - 1ull;
        const uint64_t j = n16 >> shift;
        uint32_t e = 0u;
        const uint32_t pd = checked_page(pt_d, j, dst_pages, e);
        const uint32_t ps = checked_page(pt_s, j, src_pages, e);
        if (e == 0u) {
            const uint64_t in = (n16 + threadIdx.x) & pmask;
            dst[((uint64_t)pd << shift) + in] = src[((uint64_t)ps << shift) + in];
        } else {
            raise_flag(err_word, e);
        }
    }
}

template <int U, bool EV>
__global__ __launch_bounds__(kStreamThreads) void k_relayout(
    uint8_t *__restrict__ dst, const uint32_t *__restrict__ pt_d, uint64_t dst_pages,
    const uint8_t *__restrict__ src, const uint32_t *__restrict__ pt_s, uint64_t src_pages,
    uint64_t n_bytes, uint32_t shift, uint32_t n_tiles, Gate g)
{
    constexpr uint32_t kTile = Geo<U>::kTile;
    __shared__ uint32_t s_pd[Geo<U>::kPagesMax], s_ps[Geo<U>::kPagesMax];
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t n16 = n_bytes & ~15ull;
    const uint64_t n_pages = (n16 + pmask) >> shift;
    const uint32_t lane16 = (threadIdx.x & 63u) * 16u;
    const uint32_t wbase = wave_id() * Geo<U>::kWaveSpan;
    const uint32_t *const pts[2] = {pt_d, pt_s};
    const uint64_t pools[2] = {dst_pages, src_pages};
    uint32_t *const stg[2] = {s_pd, s_ps};
    auto body = [&](uint32_t t, uint32_t, uint32_t &err, auto &&claim) {
        const uint64_t t0 = (uint64_t)t * kTile;
        const uint64_t p0 = t0 >> shift;
        stage_tile_pages<2, true>(t0, kTile, shift, n_pages, pts, pools, stg, err);
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t at = t0 + wbase + u * kStepSpan;
            const uint32_t jl = (uint32_t)((at >> shift) - p0);
            const uint32_t ps = __builtin_amdgcn_readfirstlane(s_ps[jl]);
            v[u] = buf_load_nt(chunk_rsrc(src, ps, shift, pmask, at, span_valid(at, n16, kStepSpan)),
                               lane16);
        }
        claim();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t at = t0 + wbase + u * kStepSpan;
            const uint32_t jl = (uint32_t)((at >> shift) - p0);
            const uint32_t pd = __builtin_amdgcn_readfirstlane(s_pd[jl]);
            buf_store_nt(chunk_rsrc(dst, pd, shift, pmask, at, span_valid(at, n16, kStepSpan)),
                         lane16, v[u]);
        }
        __syncthreads();
    };
    // the last n_bytes mod 16 bytes, all inside the page that holds byte n16
    auto epilogue = [&]() {
        const uint32_t rem = (uint32_t)(n_bytes - n16);
        if (threadIdx.x < rem) {
            const uint64_t j = n16 >> shift;
            uint32_t e = 0u;
            const uint32_t pd = checked_page(pt_d, j, dst_pages, e);
            const uint32_t ps = checked_page(pt_s, j, src_pages, e);
            if (e == 0u) {
                const uint64_t in = (n16 + threadIdx.x) & pmask;
                dst[((uint64_t)pd << shift) + in] = src[((uint64_t)ps << shift) + in];
            } else {
                raise_flag(g.err, e);
            }
        }
    };
    gated_tile_loop<Claim::Mid, EV>(g, n_tiles, NoOp(), body, NoOp(), epilogue);
}

// Several copies in one launch: the tiles of item i are [tile0_i,
// tile0_{i+1}); a workgroup finds the item of its tile with a scan of the
// (kernel-argument) tile offsets.
constexpr int kBatchItems = 32;
struct RelayoutItem {
    uint8_t *dst;
    const uint32_t *pt_d;
    uint64_t dst_pages;
    const uint8_t *src;
    const uint32_t *pt_s;
    uint64_t src_pages;
    uint64_t n_bytes;
    uint32_t shift;
    uint32_t tile0;  // first tile of the item
};
struct RelayoutBatch {
    RelayoutItem it[kBatchItems];
    uint32_t n;
};

template <int U>
__global__ __launch_bounds__(kStreamThreads) void k_relayout_batch(RelayoutBatch b, uint32_t n_tiles,
                                                                   Gate g)
{
    __shared__ uint32_t s_pd[Geo<U>::kPagesMax], s_ps[Geo<U>::kPagesMax];
    auto body = [&](uint32_t t, uint32_t, uint32_t &err, auto &&claim) {
        uint32_t k = 0u;
        for (uint32_t i = 1u; i < b.n; ++i)
            k = b.it[i].tile0 <= t ? i : k;
        const RelayoutItem &r = b.it[k];
        relayout_tile<U>(r.dst, r.pt_d, r.dst_pages, r.src, r.pt_s, r.src_pages, r.n_bytes,
                         r.shift, t - r.tile0, s_pd, s_ps, err, claim);
    };
    auto epilogue = [&]() {
        for (uint32_t i = 0u; i < b.n; ++i) {
            const RelayoutItem &r = b.it[i];
            relayout_tail(r.dst, r.pt_d, r.dst_pages, r.src, r.pt_s, r.src_pages, r.n_bytes,
                          r.shift, g.err);
        }
    };
    gated_tile_loop<Claim::Mid>(g, n_tiles, NoOp(), body, NoOp(), epilogue);
}

__device__ __forceinline__ u32x4 fma4(float s, u32x4 c, u32x4 b)
{
    u32x4 r;
    r.x = __float_as_uint(__builtin_fmaf(s, __uint_as_float(c.x), __uint_as_float(b.x)));
    r.y = __float_as_uint(__builtin_fmaf(s, __uint_as_float(c.y), __uint_as_float(b.y)));
    r.z = __float_as_uint(__builtin_fmaf(s, __uint_as_float(c.z), __uint_as_float(b.z)));
    r.w = __float_as_uint(__builtin_fmaf(s, __uint_as_float(c.w), __uint_as_float(b.w)));
    return r;
}

template <int U, bool EV>
__global__ __launch_bounds__(kStreamThreads) void k_triad(
    uint8_t *a, const uint32_t *__restrict__ pt_a, uint64_t a_pages,
    const uint8_t *b, const uint32_t *__restrict__ pt_b, uint64_t b_pages,
    const uint8_t *c, const uint32_t *__restrict__ pt_c, uint64_t c_pages, float s,
    uint64_t n_bytes, uint32_t shift, uint32_t n_tiles, Gate g)
{
    constexpr uint32_t kTile = Geo<U>::kTile;
    __shared__ uint32_t s_pa[Geo<U>::kPagesMax], s_pb[Geo<U>::kPagesMax], s_pc[Geo<U>::kPagesMax];
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t n16 = n_bytes & ~15ull;
    const uint64_t n_pages = (n16 + pmask) >> shift;
    const uint32_t lane16 = (threadIdx.x & 63u) * 16u;
    const uint32_t wbase = wave_id() * Geo<U>::kWaveSpan;
    const uint32_t *const pts[3] = {pt_a, pt_b, pt_c};
    const uint64_t pools[3] = {a_pages, b_pages, c_pages};
    uint32_t *const stg[3] = {s_pa, s_pb, s_pc};
    auto body = [&](uint32_t t, uint32_t, uint32_t &err, auto &&claim) {
        const uint64_t t0 = (uint64_t)t * kTile;
        const uint64_t p0 = t0 >> shift;
        // a chunk is skipped unless all three of its pages are valid
        stage_tile_pages<3, true>(t0, kTile, shift, n_pages, pts, pools, stg, err);
        u32x4 vb[U], vc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t at = t0 + wbase + u * kStepSpan;
            const uint32_t jl = (uint32_t)((at >> shift) - p0);
            const uint32_t pb = __builtin_amdgcn_readfirstlane(s_pb[jl]);
            const uint32_t pc = __builtin_amdgcn_readfirstlane(s_pc[jl]);
            const uint32_t valid = span_valid(at, n16, kStepSpan);
            vb[u] = buf_load_nt(chunk_rsrc(b, pb, shift, pmask, at, valid), lane16);
            vc[u] = buf_load_nt(chunk_rsrc(c, pc, shift, pmask, at, valid), lane16);
        }
        claim();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t at = t0 + wbase + u * kStepSpan;
            const uint32_t jl = (uint32_t)((at >> shift) - p0);
            const uint32_t pa = __builtin_amdgcn_readfirstlane(s_pa[jl]);
            buf_store_nt(chunk_rsrc(a, pa, shift, pmask, at, span_valid(at, n16, kStepSpan)),
                         lane16, fma4(s, vc[u], vb[u]));
        }
        __syncthreads();
    };
    // the last (n_bytes mod 16) / 4 elements, all inside the page of byte n16
    auto epilogue = [&]() {
        const uint32_t rem = (uint32_t)(n_bytes - n16) / 4u;
        if (threadIdx.x < rem) {
            const uint64_t j = n16 >> shift;
            uint32_t e = 0u;
            const uint32_t pa = checked_page(pt_a, j, a_pages, e);
            const uint32_t pb = checked_page(pt_b, j, b_pages, e);
            const uint32_t pc = checked_page(pt_c, j, c_pages, e);
            if (e == 0u) {
                const uint64_t in = (n16 + 4u * threadIdx.x) & pmask;
                const float r = __builtin_fmaf(s, *(const float *)(c + ((uint64_t)pc << shift) + in),
                                               *(const float *)(b + ((uint64_t)pb << shift) + in));
                *(float *)(a + ((uint64_t)pa << shift) + in) = r;
            } else {
                raise_flag(g.err, e);
            }
        }
    };
    gated_tile_loop<Claim::Mid, EV>(g, n_tiles, NoOp(), body, NoOp(), epilogue);
}

}  // namespace sgdrc

using namespace sgdrc;

extern "C" {

int bimodal_relayout(sgdrc_ctx *ctx, const sgdrc_paged *dst, const sgdrc_paged *src,
                     uint64_t n_bytes, uint32_t page_shift, void *stream)
{
    clear_error();
    int rc = check_shift(page_shift);
    if (rc)
        return rc;
    if ((rc = check_paged(dst, "dst")) || (rc = check_paged(src, "src")))
        return rc;
    Ctx *c = nullptr;
    rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    constexpr int U = kRelayoutUnroll;
    constexpr uint32_t tile = Geo<U>::kTile;
    const uint64_t n_tiles = ((n_bytes & ~15ull) + tile - 1) / tile;
    if (n_tiles >= (1ull << 31))
        return set_error(SGDRC_EINVAL, "n_bytes too large");
    const bool ev = stream_preemptible(c, stream);
    if (ev && (rc = discard_suspended(c, stream)))
        return rc;
    Gate g;
    LaunchInfo li;
    rc = make_gate(c, stream, n_tiles, kStreamGroupCus, &g, &li, ev);
    if (rc)
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    static const int occ = occupancy(k_relayout<U, false>, kStreamThreads);
    const int per_cu = std::min(occ, kStreamWgsPerCu);
    const uint32_t grid = gated_grid(c, per_cu, n_tiles, li);
    uint8_t *const d = static_cast<uint8_t *>(dst->pool);
    const uint8_t *const sp = static_cast<const uint8_t *>(src->pool);
    const uint32_t *const dpt = dst->pt, *const spt = src->pt;
    const uint64_t dpages = dst->pool_pages, spages = src->pool_pages;
    auto launch = [=](const Gate &gg, uint32_t gr, bool preempt) {
        if (preempt)
            hipLaunchKernelGGL((k_relayout<U, true>), dim3(gr), dim3(kStreamThreads), 0, s, d, dpt,
                               dpages, sp, spt, spages, n_bytes, page_shift, (uint32_t)n_tiles, gg);
        else
            hipLaunchKernelGGL((k_relayout<U, false>), dim3(gr), dim3(kStreamThreads), 0, s, d,
                               dpt, dpages, sp, spt, spages, n_bytes, page_shift,
                               (uint32_t)n_tiles, gg);
        return hipGetLastError();
    };
    SGDRC_HIP(launch(g, grid, ev));
    if (ev)
        record_preemptible(c, stream, g, n_tiles, per_cu,
                           [launch](const Gate &gg, uint32_t gr) { return launch(gg, gr, true); });
    return SGDRC_OK;
}

int bimodal_relayout_batch(sgdrc_ctx *ctx, const sgdrc_relayout_item *items, uint32_t n_items,
                           void *stream)
{
    clear_error();
    if (n_items && !items)
        return set_error(SGDRC_EINVAL, "items is NULL");
    constexpr int U = kRelayoutUnroll;
    constexpr uint32_t tile = Geo<U>::kTile;
    for (uint32_t i = 0; i < n_items; ++i) {
        const sgdrc_relayout_item &it = items[i];
        int rc = check_shift(it.page_shift);
        if (rc)
            return set_error(SGDRC_EINVAL, "item %u: page_shift %u outside [%d, %d]", i,
                             it.page_shift, SGDRC_MIN_PAGE_SHIFT, SGDRC_MAX_PAGE_SHIFT);
        if ((rc = check_paged(&it.dst, "dst")) || (rc = check_paged(&it.src, "src")))
            return set_error(SGDRC_EINVAL, "item %u: %s", i, sgdrc_last_error());
        if (it.reserved != 0)
            return set_error(SGDRC_EINVAL, "item %u: reserved must be 0", i);
        if (((it.n_bytes & ~15ull) + tile - 1) / tile >= (1ull << 31))
            return set_error(SGDRC_EINVAL, "item %u: n_bytes too large", i);
    }
    Ctx *c = nullptr;
    int rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    static const int occ = occupancy(k_relayout_batch<U>, kStreamThreads);
    const int per_cu = std::min(occ, kStreamWgsPerCu);
    for (uint32_t first = 0; first < n_items; first += kBatchItems) {
        const uint32_t n = std::min<uint32_t>(kBatchItems, n_items - first);
        RelayoutBatch b{};
        uint64_t tiles = 0;
        for (uint32_t i = 0; i < n; ++i) {
            const sgdrc_relayout_item &it = items[first + i];
            RelayoutItem &r = b.it[i];
            r.dst = static_cast<uint8_t *>(it.dst.pool);
            r.pt_d = it.dst.pt;
            r.dst_pages = it.dst.pool_pages;
            r.src = static_cast<const uint8_t *>(it.src.pool);
            r.pt_s = it.src.pt;
            r.src_pages = it.src.pool_pages;
            r.n_bytes = it.n_bytes;
            r.shift = it.page_shift;
            r.tile0 = (uint32_t)tiles;
            tiles += ((it.n_bytes & ~15ull) + tile - 1) / tile;
            if (tiles >= (1ull << 31))
                return set_error(SGDRC_EINVAL, "items %u..%u: too many bytes for one launch", first,
                                 first + i);
        }
        b.n = n;
        Gate g;
        LaunchInfo li;
        if ((rc = make_gate(c, stream, tiles, kStreamGroupCus, &g, &li, false)))
            return rc;
        const uint32_t grid = gated_grid(c, per_cu, tiles, li);
        hipLaunchKernelGGL((k_relayout_batch<U>), dim3(grid), dim3(kStreamThreads), 0, s, b,
                           (uint32_t)tiles, g);
        SGDRC_HIP(hipGetLastError());
    }
    return SGDRC_OK;
}

int colored_stream(sgdrc_ctx *ctx, const sgdrc_paged *a, const sgdrc_paged *b,
                   const sgdrc_paged *c_arr, float s, uint64_t n_elems, uint32_t page_shift,
                   void *stream)
{
    clear_error();
    int rc = check_shift(page_shift);
    if (rc)
        return rc;
    if ((rc = check_paged(a, "a")) || (rc = check_paged(b, "b")) || (rc = check_paged(c_arr, "c")))
        return rc;
    if (n_elems > (1ull << 61))
        return set_error(SGDRC_EINVAL, "n_elems too large");
    Ctx *c = nullptr;
    rc = check_ctx(ctx, &c);
    if (rc)
        return rc;
    const uint64_t n_bytes = n_elems * 4u;
    constexpr int U = kTriadUnroll, UE = kTriadUnrollEv;
    const bool ev = stream_preemptible(c, stream);
    const uint32_t tile = ev ? Geo<UE>::kTile : Geo<U>::kTile;
    const uint64_t n_tiles = ((n_bytes & ~15ull) + tile - 1) / tile;
    if (n_tiles >= (1ull << 31))
        return set_error(SGDRC_EINVAL, "n_elems too large");
    if (ev && (rc = discard_suspended(c, stream)))
        return rc;
    Gate g;
    LaunchInfo li;
    rc = make_gate(c, stream, n_tiles, kStreamGroupCus, &g, &li, ev);
    if (rc)
        return rc;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    static const int occ = occupancy(k_triad<U, false>, kStreamThreads);
    const int per_cu = std::min(occ, kStreamWgsPerCu);
    const uint32_t grid = gated_grid(c, per_cu, n_tiles, li);
    uint8_t *const ap = static_cast<uint8_t *>(a->pool);
    const uint8_t *const bp = static_cast<const uint8_t *>(b->pool);
    const uint8_t *const cp = static_cast<const uint8_t *>(c_arr->pool);
    const uint32_t *const apt = a->pt, *const bpt = b->pt, *const cpt = c_arr->pt;
    const uint64_t an = a->pool_pages, bn = b->pool_pages, cn = c_arr->pool_pages;
    auto launch = [=](const Gate &gg, uint32_t gr, bool preempt) {
        if (preempt)
            hipLaunchKernelGGL((k_triad<UE, true>), dim3(gr), dim3(kStreamThreads), 0, hs, ap, apt,
                               an, bp, bpt, bn, cp, cpt, cn, s, n_bytes, page_shift,
                               (uint32_t)n_tiles, gg);
        else
            hipLaunchKernelGGL((k_triad<U, false>), dim3(gr), dim3(kStreamThreads), 0, hs, ap, apt,
                               an, bp, bpt, bn, cp, cpt, cn, s, n_bytes, page_shift,
                               (uint32_t)n_tiles, gg);
        return hipGetLastError();
    };
    SGDRC_HIP(launch(g, grid, ev));
    if (ev)
        record_preemptible(c, stream, g, n_tiles, per_cu,
                           [launch](const Gate &gg, uint32_t gr) { return launch(gg, gr, true); });
    return SGDRC_OK;
}

}  // extern "C"
