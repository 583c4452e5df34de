// Page-table-indirected streaming kernels: bimodal relayout (page-set to
// page-set copy) and the colour-restricted triad a = b + s*c.
//
// Both run as gated persistent grids over a tile queue.  A tile is 32 KiB of
// logical bytes per array; every lane moves 8 chunks of 16 bytes
// (128 bytes in flight per lane and array) with non-temporal loads and
// stores.  When a page is at least a tile, the tile's page-table entries are
// wave-uniform scalar loads; for smaller pages the tile's entries are staged
// in LDS once per tile and every chunk looks its page up there.
#include "host_common.hpp"

namespace sgdrc {

constexpr int kStreamThreads = 256;
constexpr int kStreamUnroll = 8;
constexpr uint64_t kStreamTile = (uint64_t)kStreamThreads * 16u * kStreamUnroll;  // 32 KiB
constexpr int kStreamTileShift = 15;
constexpr int kTilePagesMax = (int)(kStreamTile >> SGDRC_MIN_PAGE_SHIFT);  // 8

// Byte-wise copy of the ragged end of a 16-byte chunk.
__device__ __forceinline__ void copy_tail(uint8_t *d, const uint8_t *s, uint32_t n)
{
    for (uint32_t i = 0; i < n; ++i)
        d[i] = s[i];
}

template <bool BIG>
__global__ __launch_bounds__(kStreamThreads) void k_relayout(
    uint8_t *__restrict__ dst, const uint32_t *__restrict__ pt_d, uint64_t dst_pages,
    const uint8_t *__restrict__ src, const uint32_t *__restrict__ pt_s, uint64_t src_pages,
    uint64_t n_bytes, uint32_t shift, uint32_t n_tiles, Gate g)
{
    __shared__ uint32_t s_pd[kTilePagesMax], s_ps[kTilePagesMax];
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t n_pages = (n_bytes + pmask) >> shift;
    auto body = [&](uint32_t t, uint32_t, uint32_t &err) {
        const uint64_t t0 = (uint64_t)t * kStreamTile;
        const uint64_t tile_bytes = n_bytes - t0 < kStreamTile ? n_bytes - t0 : kStreamTile;
        if (BIG) {
            const uint64_t j = t0 >> shift;
            const uint32_t pd = pt_d[j], ps = pt_s[j];
            const bool bad = pd >= dst_pages || ps >= src_pages;
            err |= bad ? kDevErrPtRange : 0u;
            uint8_t *d = dst + ((uint64_t)pd << shift) + (t0 & pmask);
            const uint8_t *s = src + ((uint64_t)ps << shift) + (t0 & pmask);
            if (bad) {
                // skip the tile: nothing outside the pools is touched
            } else if (tile_bytes == kStreamTile) {
                u32x4 v[kStreamUnroll];
#pragma unroll
                for (int u = 0; u < kStreamUnroll; ++u)
                    v[u] = load_nt(s + ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u);
#pragma unroll
                for (int u = 0; u < kStreamUnroll; ++u)
                    store_nt(d + ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u, v[u]);
            } else {
                for (int u = 0; u < kStreamUnroll; ++u) {
                    const uint64_t off = ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u;
                    if (off + 16u <= tile_bytes)
                        store_nt(d + off, load_nt(s + off));
                    else if (off < tile_bytes)
                        copy_tail(d + off, s + off, (uint32_t)(tile_bytes - off));
                }
            }
        } else {
            const uint64_t j0 = t0 >> shift;
            const uint32_t np = (uint32_t)(kStreamTile >> shift);
            if (threadIdx.x < np) {
                const uint64_t j = j0 + threadIdx.x;
                uint32_t pd = kBadPage, ps = kBadPage;
                if (j < n_pages) {
                    pd = checked_page(pt_d, j, dst_pages, err);
                    ps = checked_page(pt_s, j, src_pages, err);
                }
                s_pd[threadIdx.x] = pd;
                s_ps[threadIdx.x] = ps;
            }
            __syncthreads();
            u32x4 v[kStreamUnroll];
            uint8_t *dp[kStreamUnroll];
#pragma unroll
            for (int u = 0; u < kStreamUnroll; ++u) {
                const uint64_t off = ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u;
                dp[u] = nullptr;
                if (off < tile_bytes) {
                    const uint32_t jl = (uint32_t)(off >> shift);
                    const uint32_t pd = s_pd[jl], ps = s_ps[jl];
                    if (pd != kBadPage && ps != kBadPage) {
                        const uint64_t in = (t0 + off) & pmask;
                        dp[u] = dst + ((uint64_t)pd << shift) + in;
                        const uint8_t *sp = src + ((uint64_t)ps << shift) + in;
                        if (off + 16u <= tile_bytes) {
                            v[u] = load_nt(sp);
                        } else {
                            copy_tail(dp[u], sp, (uint32_t)(tile_bytes - off));
                            dp[u] = nullptr;
                        }
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kStreamUnroll; ++u)
                if (dp[u])
                    store_nt(dp[u], v[u]);
            __syncthreads();
        }
    };
    gated_tile_loop<false>(g, n_tiles, body, NoOp(), NoOp());
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

template <bool BIG>
__global__ __launch_bounds__(kStreamThreads) void k_triad(
    uint8_t *a, const uint32_t *__restrict__ pt_a, uint64_t a_pages,
    const uint8_t *b, const uint32_t *__restrict__ pt_b, uint64_t b_pages,
    const uint8_t *c, const uint32_t *__restrict__ pt_c, uint64_t c_pages, float s,
    uint64_t n_bytes, uint32_t shift, uint32_t n_tiles, Gate g)
{
    __shared__ uint32_t s_pa[kTilePagesMax], s_pb[kTilePagesMax], s_pc[kTilePagesMax];
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t n_pages = (n_bytes + pmask) >> shift;
    auto body = [&](uint32_t t, uint32_t, uint32_t &err) {
        const uint64_t t0 = (uint64_t)t * kStreamTile;
        const uint64_t tile_bytes = n_bytes - t0 < kStreamTile ? n_bytes - t0 : kStreamTile;
        if (BIG) {
            const uint64_t j = t0 >> shift;
            const uint32_t pa = pt_a[j], pb = pt_b[j], pc = pt_c[j];
            const bool bad = pa >= a_pages || pb >= b_pages || pc >= c_pages;
            err |= bad ? kDevErrPtRange : 0u;
            const uint64_t in = t0 & pmask;
            uint8_t *ap = a + ((uint64_t)pa << shift) + in;
            const uint8_t *bp = b + ((uint64_t)pb << shift) + in;
            const uint8_t *cp = c + ((uint64_t)pc << shift) + in;
            if (bad) {
                // skip the tile: nothing outside the pools is touched
            } else if (tile_bytes == kStreamTile) {
                u32x4 vb[kStreamUnroll], vc[kStreamUnroll];
#pragma unroll
                for (int u = 0; u < kStreamUnroll; ++u) {
                    const uint64_t off = ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u;
                    vb[u] = load_nt(bp + off);
                    vc[u] = load_nt(cp + off);
                }
#pragma unroll
                for (int u = 0; u < kStreamUnroll; ++u) {
                    const uint64_t off = ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u;
                    store_nt(ap + off, fma4(s, vc[u], vb[u]));
                }
            } else {
                for (int u = 0; u < kStreamUnroll; ++u) {
                    const uint64_t off = ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u;
                    if (off + 16u <= tile_bytes) {
                        store_nt(ap + off, fma4(s, load_nt(cp + off), load_nt(bp + off)));
                    } else if (off < tile_bytes) {
                        for (uint64_t e = off; e < tile_bytes; e += 4) {
                            const float r = __builtin_fmaf(s, *(const float *)(cp + e),
                                                           *(const float *)(bp + e));
                            *(float *)(ap + e) = r;
                        }
                    }
                }
            }
        } else {
            const uint64_t j0 = t0 >> shift;
            const uint32_t np = (uint32_t)(kStreamTile >> shift);
            if (threadIdx.x < np) {
                const uint64_t j = j0 + threadIdx.x;
                uint32_t pa = kBadPage, pb = kBadPage, pc = kBadPage;
                if (j < n_pages) {
                    pa = checked_page(pt_a, j, a_pages, err);
                    pb = checked_page(pt_b, j, b_pages, err);
                    pc = checked_page(pt_c, j, c_pages, err);
                }
                s_pa[threadIdx.x] = pa;
                s_pb[threadIdx.x] = pb;
                s_pc[threadIdx.x] = pc;
            }
            __syncthreads();
            u32x4 vb[kStreamUnroll], vc[kStreamUnroll];
            uint8_t *ap[kStreamUnroll];
#pragma unroll
            for (int u = 0; u < kStreamUnroll; ++u) {
                const uint64_t off = ((uint64_t)u * kStreamThreads + threadIdx.x) * 16u;
                ap[u] = nullptr;
                if (off < tile_bytes) {
                    const uint32_t jl = (uint32_t)(off >> shift);
                    const uint32_t pa = s_pa[jl], pb = s_pb[jl], pc = s_pc[jl];
                    if (pa != kBadPage && pb != kBadPage && pc != kBadPage) {
                        const uint64_t in = (t0 + off) & pmask;
                        uint8_t *aq = a + ((uint64_t)pa << shift) + in;
                        const uint8_t *bq = b + ((uint64_t)pb << shift) + in;
                        const uint8_t *cq = c + ((uint64_t)pc << shift) + in;
                        if (off + 16u <= tile_bytes) {
                            vb[u] = load_nt(bq);
                            vc[u] = load_nt(cq);
                            ap[u] = aq;
                        } else {
                            for (uint64_t e = 0; e < tile_bytes - off; e += 4) {
                                const float r = __builtin_fmaf(s, *(const float *)(cq + e),
                                                               *(const float *)(bq + e));
                                *(float *)(aq + e) = r;
                            }
                        }
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kStreamUnroll; ++u)
                if (ap[u])
                    store_nt(ap[u], fma4(s, vc[u], vb[u]));
            __syncthreads();
        }
    };
    gated_tile_loop<false>(g, n_tiles, body, NoOp(), NoOp());
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
    const uint64_t n_tiles = (n_bytes + kStreamTile - 1) / kStreamTile;
    if (n_tiles >= (1ull << 31))
        return set_error(SGDRC_EINVAL, "n_bytes too large");
    Gate g;
    LaunchInfo li;
    rc = make_gate(c, stream, n_tiles, kStreamGroupCus, &g, &li);
    if (rc)
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool big = page_shift >= kStreamTileShift;
    static const int occ_big = occupancy(k_relayout<true>, kStreamThreads);
    static const int occ_small = occupancy(k_relayout<false>, kStreamThreads);
    const uint32_t grid = gated_grid(c, big ? occ_big : occ_small, n_tiles, li);
    auto kern = big ? k_relayout<true> : k_relayout<false>;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kStreamThreads), 0, s,
                       static_cast<uint8_t *>(dst->pool), dst->pt, dst->pool_pages,
                       static_cast<const uint8_t *>(src->pool), src->pt, src->pool_pages, n_bytes,
                       page_shift, (uint32_t)n_tiles, g);
    SGDRC_HIP(hipGetLastError());
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
    const uint64_t n_tiles = (n_bytes + kStreamTile - 1) / kStreamTile;
    if (n_tiles >= (1ull << 31))
        return set_error(SGDRC_EINVAL, "n_elems too large");
    Gate g;
    LaunchInfo li;
    rc = make_gate(c, stream, n_tiles, kStreamGroupCus, &g, &li);
    if (rc)
        return rc;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    const bool big = page_shift >= kStreamTileShift;
    static const int occ_big = occupancy(k_triad<true>, kStreamThreads);
    static const int occ_small = occupancy(k_triad<false>, kStreamThreads);
    const uint32_t grid = gated_grid(c, big ? occ_big : occ_small, n_tiles, li);
    auto kern = big ? k_triad<true> : k_triad<false>;
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kStreamThreads), 0, hs,
                       static_cast<uint8_t *>(a->pool), a->pt, a->pool_pages,
                       static_cast<const uint8_t *>(b->pool), b->pt, b->pool_pages,
                       static_cast<const uint8_t *>(c_arr->pool), c_arr->pt, c_arr->pool_pages, s,
                       n_bytes, page_shift, (uint32_t)n_tiles, g);
    SGDRC_HIP(hipGetLastError());
    return SGDRC_OK;
}

}  // extern "C"
