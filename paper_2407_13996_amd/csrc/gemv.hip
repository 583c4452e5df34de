// Colour-restricted GEMV / small-batch GEMM: y[b][m] = sum_k W[m][k] x[b][k].
//
// W is row-major [M x K] in a paged pool and is streamed once from HBM with
// 16-byte non-temporal loads; x and y are small and contiguous.  A tile is a
// block of whole rows, so each output is produced by exactly one workgroup
// in a fixed summation order: per-lane fp32 FMA chains over that lane's
// 16-byte slices of the row, a butterfly over the 64 lanes, then the four
// waves' partials added in wave order.  The result therefore depends only on
// (M, K, batch, dtypes) and not on which CUs ran the tiles.
//
// Page translation: the page-table entries covering a tile's rows are staged
// in LDS at the start of the tile (at most kPtCap; beyond that each lane
// reads the table directly), and every 16-byte slice is mapped with one LDS
// read plus a shift and an add.
//
// Batches 3..8 with bf16 x bf16 or f16 x f16 operands use the gfx950
// 16x16x32 MFMA: a 16-row block of W is the A operand, x (batch padded to 16
// columns) the B operand; eight wavefronts split each chunk of K.  From batch
// 3 on it measured faster than the vector path on MI355X.
#include "host_common.hpp"

namespace sgdrc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

constexpr int kGemvThreads = 256;
constexpr int kGemvWaves = kGemvThreads / 64;
constexpr int kGemvRowsMax = 4;  // rows per tile, vector-ALU path (at most)
constexpr int kMfmaRows = 16;    // rows per tile, MFMA path
// MFMA path: 8 waves split K, so that a 16-row tile keeps twice the loads of
// a 4-wave workgroup in flight (measured best of 4, 8 and 16 waves for both
// 4096x11008 and 11008x4096 at batch 8)
constexpr int kMfmaThreads = 512;
constexpr int kMfmaWaves = kMfmaThreads / 64;
constexpr int kPtCap = 256;      // page-table entries staged per tile (one per thread)

template <int DT> struct Dt;
template <> struct Dt<SGDRC_F32> { static constexpr int size = 4; };
template <> struct Dt<SGDRC_BF16> { static constexpr int size = 2; };
template <> struct Dt<SGDRC_F16> { static constexpr int size = 2; };

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }
__device__ __forceinline__ float f16_lo(uint32_t v)
{
    return (float)__builtin_bit_cast(f16x2, v).x;
}
__device__ __forceinline__ float f16_hi(uint32_t v)
{
    return (float)__builtin_bit_cast(f16x2, v).y;
}

// Decode N elements of type DT held in the words w[0..] into f[0..N).
template <int DT, int N>
__device__ __forceinline__ void decode(const uint32_t *w, float *f)
{
    if (DT == SGDRC_F32) {
#pragma unroll
        for (int i = 0; i < N; ++i)
            f[i] = __uint_as_float(w[i]);
    } else if (DT == SGDRC_BF16) {
#pragma unroll
        for (int i = 0; i < N / 2; ++i) {
            f[2 * i] = bf16_lo(w[i]);
            f[2 * i + 1] = bf16_hi(w[i]);
        }
    } else {
#pragma unroll
        for (int i = 0; i < N / 2; ++i) {
            f[2 * i] = f16_lo(w[i]);
            f[2 * i + 1] = f16_hi(w[i]);
        }
    }
}

// Page-table entries of one tile, staged in LDS.  The host guarantees that
// a tile spans at most kPtCap pages.
struct TilePages {
    uint64_t p_lo;
};

__device__ __forceinline__ TilePages stage_pages(const uint32_t *pt, uint64_t pool_pages,
                                                 uint64_t byte_lo, uint64_t byte_hi,
                                                 uint32_t shift, uint32_t *s_pt, uint32_t &err)
{
    TilePages tp;
    tp.p_lo = byte_lo >> shift;
    const uint32_t np = (uint32_t)(((byte_hi - 1) >> shift) - tp.p_lo + 1);
    if (threadIdx.x < np)
        s_pt[threadIdx.x] = checked_page(pt, tp.p_lo + threadIdx.x, pool_pages, err);
    __syncthreads();
    return tp;
}

__device__ __forceinline__ uint32_t page_of(const TilePages &tp, const uint32_t *s_pt, uint64_t j)
{
    return s_pt[j - tp.p_lo];
}

// When the whole matrix spans at most kPtCap pages, its table is staged in
// LDS once per workgroup, in the tile loop's prologue (overlapping the
// gate's own reads), and tiles skip their per-tile staging.  The staging is
// straight-line: threads beyond the last page read and write that page's
// entry again.  Out-of-range entries are recorded in ``err``.
__device__ __forceinline__ void stage_whole_table(const uint32_t *pt, uint64_t pool_pages,
                                                  uint64_t w_pages, uint32_t *s_pt, uint32_t &err)
{
    const uint64_t n = w_pages < (uint64_t)kPtCap ? w_pages : (uint64_t)kPtCap;
    const uint32_t i = threadIdx.x < n ? threadIdx.x : (uint32_t)(n - 1u);
    uint32_t e = 0u;
    s_pt[i] = checked_page(pt, i, pool_pages, e);
    err |= threadIdx.x < n ? e : 0u;
}

// Page lookup context of one tile: the whole staged table, or this tile's
// pages staged now (a barrier; the choice is uniform).
__device__ __forceinline__ TilePages tile_pages(bool whole, const uint32_t *pt, uint64_t pool_pages,
                                                uint64_t byte_lo, uint64_t byte_hi, uint32_t shift,
                                                uint32_t *s_pt, uint32_t &err)
{
    if (whole)
        return TilePages{0u};
    return stage_pages(pt, pool_pages, byte_lo, byte_hi, shift, s_pt, err);
}

// R rows per tile; U 16-byte slices per lane and row in flight; XO: x is
// loaded once per workgroup (the host sets it only for rows that one round
// of loads covers).
template <int WT, int XT, int NB, int R, int U, bool XO>
__global__ __launch_bounds__(kGemvThreads) void k_gemv_valu(
    const uint8_t *__restrict__ w_pool, const uint32_t *__restrict__ pt, uint64_t pool_pages,
    uint32_t M, uint32_t K, const uint8_t *__restrict__ x, uint32_t nb, float *__restrict__ y,
    uint32_t shift, uint32_t n_tiles, Gate g)
{
    constexpr int WSZ = Dt<WT>::size, XSZ = Dt<XT>::size;
    constexpr int EPV = 16 / WSZ;                 // elements per 16-byte slice of W
    constexpr int XW = EPV * XSZ / 4;             // 32-bit words of x per slice and batch
    __shared__ uint32_t s_pt[kPtCap];
    __shared__ float s_red[kGemvWaves][R * NB];
    const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63u;
    const uint64_t row_bytes = (uint64_t)K * WSZ;
    const uint32_t KV = (uint32_t)(row_bytes / 16u);
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t w_pages = ((uint64_t)M * row_bytes + pmask) >> shift;
    const bool whole = w_pages <= (uint64_t)kPtCap;
    uint32_t pro_err = 0u;
    // x of slice kv for every batch row (zeros out of range)
    auto load_x = [&](uint32_t kv, uint32_t (&xs)[NB][XW]) __attribute__((always_inline)) {
        const bool ok = kv < KV;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
#pragma unroll
            for (int i = 0; i < XW; ++i)
                xs[b][i] = 0u;
            if (ok && (uint32_t)b < nb) {
                const uint8_t *xp = x + ((uint64_t)b * K + (uint64_t)kv * EPV) * XSZ;
                if (XW == 2) {
                    u32x2 v = *reinterpret_cast<const u32x2 *>(xp);
                    xs[b][0] = v.x;
                    xs[b][1] = v.y;
                } else {
#pragma unroll
                    for (int q = 0; q < XW / 4; ++q) {
                        u32x4 v = *reinterpret_cast<const u32x4 *>(xp + 16 * q);
                        xs[b][4 * q + 0] = v.x;
                        xs[b][4 * q + 1] = v.y;
                        xs[b][4 * q + 2] = v.z;
                        xs[b][4 * q + 3] = v.w;
                    }
                }
            }
        }
    };
    // XO (a row that one round of loads covers): every tile uses the same
    // x slices per lane, loaded once per workgroup and kept in registers.
    constexpr bool x_once = XO;
    uint32_t xk[U][NB][XW];
    auto prologue = [&]() {
        stage_whole_table(pt, pool_pages, w_pages, s_pt, pro_err);
        if (x_once) {
#pragma unroll
            for (int u = 0; u < U; ++u)
                load_x((uint32_t)(u * kGemvWaves) * 64u + wave * 64u + lane, xk[u]);
        }
    };

    auto body = [&](uint32_t t, uint32_t, uint32_t &err, auto &&) {
        const uint32_t m0 = t * R;
        const uint32_t m_end = min(m0 + (uint32_t)R, M);
        const TilePages tp = tile_pages(whole, pt, pool_pages, (uint64_t)m0 * row_bytes,
                                        (uint64_t)m_end * row_bytes, shift, s_pt, err);
        float acc[R][NB];
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int b = 0; b < NB; ++b)
                acc[r][b] = 0.0f;

        for (uint32_t j = 0; (j * kGemvWaves + wave) * 64u < KV; j += U) {
            u32x4 wv[U][R];
            uint32_t xl[U][NB][XW];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t kv = ((j + u) * kGemvWaves + wave) * 64u + lane;
                const bool ok = kv < KV;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    wv[u][r] = u32x4{0u, 0u, 0u, 0u};
                    if (ok && m0 + r < M) {
                        const uint64_t off = (uint64_t)(m0 + r) * row_bytes + (uint64_t)kv * 16u;
                        const uint32_t p = page_of(tp, s_pt, off >> shift);
                        if (p != kBadPage)
                            wv[u][r] = load_nt(w_pool + ((uint64_t)p << shift) + (off & pmask));
                    }
                }
                if (!x_once)
                    load_x(kv, xl[u]);
            }
            const uint32_t (&xv)[U][NB][XW] = x_once ? xk : xl;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float xf[NB][EPV];
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    decode<XT, EPV>(xv[u][b], xf[b]);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const uint32_t ww[4] = {wv[u][r].x, wv[u][r].y, wv[u][r].z, wv[u][r].w};
                    float wf[EPV];
                    decode<WT, EPV>(ww, wf);
#pragma unroll
                    for (int e = 0; e < EPV; ++e)
#pragma unroll
                        for (int b = 0; b < NB; ++b)
                            acc[r][b] = __builtin_fmaf(wf[e], xf[b][e], acc[r][b]);
                }
            }
        }
        // butterfly over the 64 lanes: every lane ends with the same sum
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                float v = acc[r][b];
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1)
                    v += __shfl_xor(v, off, 64);
                acc[r][b] = v;
            }
        if (lane == 0) {
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    s_red[wave][r * NB + b] = acc[r][b];
        }
        __syncthreads();
        if (threadIdx.x < (uint32_t)(R * NB)) {
            const uint32_t r = threadIdx.x / NB, b = threadIdx.x % NB;
            float v = s_red[0][threadIdx.x];
#pragma unroll
            for (int w = 1; w < kGemvWaves; ++w)
                v += s_red[w][threadIdx.x];
            if (b < nb && m0 + r < M)
                y[(uint64_t)b * M + m0 + r] = v;
        }
        __syncthreads();
    };
    tile_loop<Claim::Ahead>(g, n_tiles, prologue, body);
    if (pro_err)
        raise_flag(g.err, pro_err);
}

template <int DT>
__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c)
{
    if (DT == SGDRC_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                       __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                      __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// Batch 3..8 on MFMA.  A tile (16 or 8 rows x K) is consumed in chunks of
// kMfmaChunk bytes per row.  Each chunk of W (the tile's rows) and of x (XB =
// 4 or 8 batch rows: the batch rounded up) is read with row-contiguous
// 16-byte loads (each wavefront
// instruction covers 1 KiB of one row) and staged in LDS; the MFMAs then
// read their operands from LDS: lane l supplies row (l % 16) of the W block
// and batch column (l % 16) of x, both for the 16-byte k-slice of its lane
// group g = l / 16, so the k order inside the instruction matches between
// the operands, and the accumulator holds rows 4g..4g+3 of batch column
// l % 16.  The eight waves take the chunk's 32 k-steps four each.  The
// kMfmaSets chunks that follow are in flight during the current chunk's
// MFMAs; beyond the last chunk the loads read a valid address and are
// discarded.  Two sets keep two workgroups per CU (three or more need
// more than 128 VGPRs and measured slower).  Batch columns past XB are
// zero in the B operand; a column's sums do not depend on the others, so
// XB does not change a result.  Staging 4 x rows instead of 8 at batch 3
// and 4 halves the x loads and LDS writes: 2-6.6 percent faster over the
// bf16 4096 x 11008 and 11008 x 4096 layers on 64..256 CUs (two
// interleaved runs, same box).
constexpr uint32_t kMfmaChunk = 2048;                  // bytes per row per chunk
constexpr uint32_t kMfmaChunkSlices = kMfmaChunk / 16u;  // 128
constexpr uint32_t kMfmaLdsRow = kMfmaChunk + 16u;     // padded LDS row
constexpr int kMfmaBatchRows = 8;                      // x rows staged at most (batch <= 8)
constexpr int kMfmaStepsPerWave = (int)(kMfmaChunk / 64u) / kMfmaWaves;             // 4
constexpr int kMfmaSets = 2;  // register sets of chunk loads in flight

// x through a buffer resource, cached (every workgroup reads all of x).
constexpr uint32_t kXOutside = 0xFFFFFFF0u;  // offset past any x resource
__device__ __forceinline__ u32x4 buf_load(Rsrc r, uint32_t off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// A row of W through its own buffer resource, for tiles that lie inside one
// page (the common case: a 2 MiB page holds many tiles): base = the row's
// first byte in the pool, range = the row's bytes, or 0 for a row past M or
// a page-table entry outside the pool.  Loads then take the lane's offset in
// the row and read zeros past it, with no table read, select or branch per
// load.
__device__ __forceinline__ Rsrc row_rsrc(uint64_t phys_row, bool valid, uint64_t row_bytes)
{
    return make_rsrc(reinterpret_cast<const void *>(phys_row), valid ? (uint32_t)row_bytes : 0u);
}

// The physical address of a tile's first byte when the tile lies inside
// one page (the entry of that page; a bad entry is reported by the caller's
// validity test), made wave-uniform so that resources built from it live in
// scalar registers.
__device__ __forceinline__ uint64_t tile_phys(const uint8_t *w_pool, uint32_t entry, uint64_t t_lo,
                                              uint32_t shift, uint64_t pmask)
{
    const uint64_t a = reinterpret_cast<uint64_t>(w_pool) + ((uint64_t)entry << shift) + (t_lo & pmask);
    // (the builtin returns int: each half goes through uint32_t, so that
    // the low half is not sign-extended into the high one)
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return (uint64_t)lo | (uint64_t)hi << 32;
}

// XA: x is staged for the whole K in LDS once per workgroup (rows of at
// most kXaBytes) instead of chunk by chunk; chunks past the end (pads) are
// then skipped rather than multiplied by zeros.  The sum starts at +0 and
// every added partial is a sum of exact products, so it can never become
// -0: skipping a pad's +0 leaves the same bits.
constexpr uint32_t kXaBytes = 8192u;
template <int DT, int ROWS, int XB, bool XA>
__global__ __launch_bounds__(kMfmaThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_gemm_mfma(
    const uint8_t *__restrict__ w_pool, const uint32_t *__restrict__ pt, uint64_t pool_pages,
    uint32_t M, uint32_t K, const uint8_t *__restrict__ x, uint32_t nb, float *__restrict__ y,
    uint32_t shift, uint32_t n_tiles, Gate g)
{
    __shared__ uint32_t s_pt[kPtCap];
    __shared__ f32x4 s_red[kMfmaWaves][64];
    // ROWS = 16 fills the MFMA's A operand; ROWS = 8 leaves its upper half
    // zero (twice the tiles, for masks with few tiles per CU).  An output's
    // sum does not depend on the other rows of its tile, so both give the
    // same bits.
    static_assert(ROWS == 16 || ROWS == 8, "tiles of 16 or 8 rows");
    constexpr int WL = ROWS * (int)kMfmaChunkSlices / kMfmaThreads;  // W loads per lane
    __shared__ __attribute__((aligned(16))) uint8_t s_w[ROWS][kMfmaLdsRow];
    static_assert(XB == 4 || XB == kMfmaBatchRows, "4 or 8 x rows");
    constexpr int XL = XB * (int)kMfmaChunkSlices / kMfmaThreads;  // x loads per lane (1 or 2)
    __shared__ __attribute__((aligned(16))) uint8_t s_x[XA ? 1 : XB][XA ? 16 : kMfmaLdsRow];
    __shared__ __attribute__((aligned(16))) uint8_t s_xa[XA ? XB : 1][XA ? kXaBytes + 16u : 16u];
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t rl = lane & 15u, grp = lane >> 4;
    const uint64_t row_bytes = (uint64_t)K * 2u;
    const uint32_t KV = (uint32_t)(row_bytes / 16u);
    const uint32_t n_chunks = (KV + kMfmaChunkSlices - 1u) / kMfmaChunkSlices;
    const uint64_t pmask = (1ull << shift) - 1ull;
    const uint64_t w_pages = ((uint64_t)M * row_bytes + pmask) >> shift;
    const bool whole = w_pages <= (uint64_t)kPtCap;
    // x is below 4 GiB (checked by the host), so 32-bit offsets reach it
    const uint32_t x_row = K * 2u;
    const Rsrc x_rsrc = make_rsrc(x, nb * x_row);
    uint32_t pro_err = 0u;
    auto prologue = [&]() {
        stage_whole_table(pt, pool_pages, w_pages, s_pt, pro_err);
        if (XA) {
            constexpr uint32_t kSl = kXaBytes / 16u;
#pragma unroll
            for (int q = 0; q < XB * (int)kSl / kMfmaThreads; ++q) {
                const uint32_t i = (uint32_t)q * kMfmaThreads + threadIdx.x;
                const uint32_t b = i / kSl, sl = i % kSl;
                *reinterpret_cast<u32x4 *>(&s_xa[b][sl * 16u]) =
                    buf_load(x_rsrc, b < nb && sl < KV ? b * x_row + sl * 16u : kXOutside);
            }
        }
    };

    auto body = [&](uint32_t t, uint32_t, uint32_t &err, auto &&) {
        const uint32_t m0 = t * (uint32_t)ROWS;
        const uint32_t m_end = min(m0 + (uint32_t)ROWS, M);
        const TilePages tp = tile_pages(whole, pt, pool_pages, (uint64_t)m0 * row_bytes,
                                        (uint64_t)m_end * row_bytes, shift, s_pt, err);
        // kMfmaSets register sets of chunk loads, so that that many chunks are
        // in flight while another feeds the MFMAs.  Loads are always issued
        // and are zero where out of range (rows beyond M, slices beyond K,
        // batch rows beyond nb), so chunks are taken kMfmaSets at a time
        // without a branch; pad chunks past the end add zeros.
        // The in-range test of each load travels beside its data as a bit of
        // ``okv`` and is applied where the data goes to LDS: a select right
        // after the load would make the loop wait for the data there.
        // The rows of 16-row block b = m0 / 16 walk their chunks starting at
        // chunk b mod n_chunks (then wrapping), so that the workgroups
        // streaming at one moment read different offsets of their rows
        // instead of all the same one.  On MI355X (the bf16 4096 x 11008
        // and 11008 x 4096 layers in 2 MiB pages, batch 4 and 8, same session): 2.3-4.2 percent faster on
        // 256 CUs, up to 6.9 percent on 192, up to 1.6 percent slower at
        // batch 8 on 64 CUs, where each CU streams several tiles and the
        // wrap splits each row in two runs; walking odd blocks backwards
        // instead gained nothing.  The order depends on the rows only (an 8-row tile takes
        // the order of the 16-row block it lies in), so neither the tile
        // height nor the CU mask changes a result.
        const uint32_t rot = __builtin_amdgcn_readfirstlane((m0 / 16u) % n_chunks);
        f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        // The chunk loop, with W read by ``load_w(c, q, okv)``: load q of
        // this lane in chunk c, which sets bit q of ``okv`` when its data is
        // valid.
        auto run = [&](auto &&load_w) __attribute__((always_inline)) {
            // ``cl``: the chunk's place in the tile's order; past n_chunks a pad
            auto load_chunk = [&](uint32_t cl, u32x4 *wv, u32x4 *xv, uint32_t &okv) __attribute__((always_inline)) {
                const uint32_t c = __builtin_amdgcn_readfirstlane(
                    cl >= n_chunks ? n_chunks : (cl + rot >= n_chunks ? cl + rot - n_chunks : cl + rot));
                okv = 0u;
#pragma unroll
                for (int q = 0; q < WL; ++q)
                    wv[q] = load_w(c, q, okv);
#pragma unroll
                for (int q = 0; q < (XA ? 0 : XL); ++q) {
                    const uint32_t L = (uint32_t)q * kMfmaThreads + threadIdx.x;
                    const uint32_t b = L / kMfmaChunkSlices, sl = L % kMfmaChunkSlices;
                    const uint32_t kv = c * kMfmaChunkSlices + sl;
                    // out of range: an offset beyond the resource, which reads zero
                    xv[q] = buf_load(x_rsrc, b < nb && kv < KV ? b * x_row + kv * 16u : kXOutside);
                }
            };
            auto store_chunk = [&](const u32x4 *wv, const u32x4 *xv, uint32_t okv) __attribute__((always_inline)) {
                const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int q = 0; q < WL; ++q) {
                    const uint32_t L = (uint32_t)q * kMfmaThreads + threadIdx.x;
                    *reinterpret_cast<u32x4 *>(&s_w[L / kMfmaChunkSlices][(L % kMfmaChunkSlices) * 16u]) =
                        (okv >> q) & 1u ? wv[q] : z;
                }
#pragma unroll
                for (int q = 0; q < (XA ? 0 : XL); ++q) {
                    const uint32_t L = (uint32_t)q * kMfmaThreads + threadIdx.x;
                    *reinterpret_cast<u32x4 *>(&s_x[L / kMfmaChunkSlices][(L % kMfmaChunkSlices) * 16u]) = xv[q];
                }
            };
            auto mfma_chunk = [&](uint32_t cx) __attribute__((always_inline)) {
#pragma unroll
                for (int i = 0; i < kMfmaStepsPerWave; ++i) {
                    const uint32_t j = wave * (uint32_t)kMfmaStepsPerWave + (uint32_t)i;
                    const u32x4 a = *reinterpret_cast<const u32x4 *>(
                        &s_w[rl & (uint32_t)(ROWS - 1)][j * 64u + grp * 16u]);
                    const u32x4 bx = XA ? *reinterpret_cast<const u32x4 *>(
                                              &s_xa[rl & (uint32_t)(XB - 1)][cx * kMfmaChunk + j * 64u + grp * 16u])
                                        : *reinterpret_cast<const u32x4 *>(
                                              &s_x[XA ? 0u : (rl & (uint32_t)(XB - 1))][XA ? 0u : j * 64u + grp * 16u]);
                    const u32x4 z = {0u, 0u, 0u, 0u};
                    acc = mfma16x16x32<DT>(rl < (uint32_t)ROWS ? a : z,
                                           rl < (uint32_t)XB ? bx : z, acc);
                }
            };
            u32x4 ws[kMfmaSets][WL], xs[kMfmaSets][XL];
            uint32_t oks[kMfmaSets];
#pragma unroll
            for (int s = 0; s < kMfmaSets; ++s)
                load_chunk((uint32_t)s, ws[s], xs[s], oks[s]);
            for (uint32_t c = 0; c < n_chunks; c += (uint32_t)kMfmaSets) {
#pragma unroll
                for (int s = 0; s < kMfmaSets; ++s) {
                    __syncthreads();  // the previous chunk's MFMAs have read the LDS
                    store_chunk(ws[s], xs[s], oks[s]);
                    __syncthreads();
                    load_chunk(c + (uint32_t)(kMfmaSets + s), ws[s], xs[s], oks[s]);
                    {
                        // the consumed chunk's index (x of a pad chunk is not staged: skipped)
                        const uint32_t cl = c + (uint32_t)s;
                        const uint32_t cx = __builtin_amdgcn_readfirstlane(
                            cl + rot >= n_chunks ? cl + rot - n_chunks : cl + rot);
                        if (!XA || cl < n_chunks)
                            mfma_chunk(cx);
                    }
                }
            }
        };
        // A lane's W loads share its 16-byte slice of the chunk (the grid of
        // loads is kMfmaThreads wide, a whole number of chunk rows) and step
        // by kRowStep rows; a chunk row is a whole number of wavefronts, so
        // a wave's loads q all read one row.
        static_assert(kMfmaThreads % kMfmaChunkSlices == 0 && kMfmaChunkSlices % 64u == 0,
                      "loads cover whole chunk rows, a row per wave");
        constexpr uint32_t kRowStep = kMfmaThreads / kMfmaChunkSlices;
        const uint32_t w_sl = threadIdx.x % kMfmaChunkSlices;
        const uint32_t w_r = __builtin_amdgcn_readfirstlane(threadIdx.x / kMfmaChunkSlices);
        const uint64_t t_lo = (uint64_t)m0 * row_bytes, t_hi = (uint64_t)m_end * row_bytes;
        if ((t_lo >> shift) == ((t_hi - 1u) >> shift)) {
            // the tile lies inside one page: a buffer resource per row; past
            // the row (pad chunks, slices beyond K) the loads read zeros.
            // On MI355X (bf16 4096 x 11008 and 11008 x 4096 in 2 MiB pages,
            // batch 4 and 8, 64..256 CUs, same session): 2.1 percent faster
            // on average than a table read per load, up to 6 percent on
            // 11008 x 4096.  The same change in the vector-ALU kernel was
            // 2-3 percent slower at batch 1, so that kernel keeps its
            // per-load lookups.
            const uint32_t e = __builtin_amdgcn_readfirstlane(page_of(tp, s_pt, t_lo >> shift));
            const uint64_t phys = tile_phys(w_pool, e, t_lo, shift, pmask);
            Rsrc rr[WL];
#pragma unroll
            for (int q = 0; q < WL; ++q) {
                const uint32_t r = w_r + (uint32_t)q * kRowStep;
                rr[q] = row_rsrc(phys + (uint64_t)r * row_bytes, e != kBadPage && m0 + r < M, row_bytes);
            }
            run([&](uint32_t c, int q, uint32_t &okv) __attribute__((always_inline)) {
                okv |= 1u << q;
                return buf_load_nt(rr[q], c * kMfmaChunk + w_sl * 16u);
            });
        } else {
            // the tile crosses a page boundary: a table read per load
            const uint64_t w_base = (uint64_t)(m0 + w_r) * row_bytes + (uint64_t)w_sl * 16u;
            run([&](uint32_t c, int q, uint32_t &okv) __attribute__((always_inline)) {
                const bool in = c * kMfmaChunkSlices + w_sl < KV && m0 + w_r + (uint32_t)q * kRowStep < M;
                // out of range: the tile's first byte (a valid page), data discarded
                const uint64_t off = in ? w_base + (uint64_t)q * kRowStep * row_bytes + (uint64_t)c * kMfmaChunk
                                        : t_lo;
                const uint32_t p = page_of(tp, s_pt, off >> shift);
                const bool ok = in && p != kBadPage;
                okv |= (uint32_t)ok << q;
                return load_nt(w_pool + (ok ? ((uint64_t)p << shift) + (off & pmask) : 0u));
            });
        }
        s_red[wave][lane] = acc;
        __syncthreads();
        if (wave == 0) {
            f32x4 v = s_red[0][lane];
#pragma unroll
            for (int w = 1; w < kMfmaWaves; ++w) {
                f32x4 o = s_red[w][lane];
                v.x += o.x;
                v.y += o.y;
                v.z += o.z;
                v.w += o.w;
            }
            if (rl < nb) {
                const float vals[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t m = m0 + grp * 4u + (uint32_t)i;
                    if (m < m_end)
                        y[(uint64_t)rl * M + m] = vals[i];
                }
            }
        }
        __syncthreads();
    };
    tile_loop<Claim::Ahead>(g, n_tiles, prologue, body);
    if (pro_err)
        raise_flag(g.err, pro_err);
}

typedef void (*GemvKernel)(const uint8_t *, const uint32_t *, uint64_t, uint32_t, uint32_t,
                           const uint8_t *, uint32_t, float *, uint32_t, uint32_t, Gate);

static int dtype_size(int dt) { return dt == SGDRC_F32 ? 4 : 2; }

// The launch plan of colored_gemv: which kernel, tile height and loads in
// flight, decided from the shape and the number of CUs the mask allows.
// Vector-ALU path, measured on MI355X over the 4096x11008 and 11008x4096
// bf16 layers under the static schedule (masks of 64..256 CUs, eight
// rotated weight copies): four-row tiles, the whole row in flight per lane
// where it fits (two 16-byte loads per lane and row for rows of 8 KiB,
// three for longer ones), except batch 1 with long rows when each allowed CU
// has few tiles (``few``): the kernel is then bound by the latency of one
// tile, and two-row tiles that load a 22 KB row in one round (six loads per
// lane) finish sooner (4096 x 11008 on 256 CUs 15.1 against 15.2 us, on 192
// CUs 17.9 against 18.9 us); with many tiles per CU, four-row tiles won (64
// CUs 38.4 against 42.2 us) until x was loaded once per workgroup (below):
// with that, two-row tiles over one round of loads win on every mask for
// rows of W and x of one type (4096 x 11008 on 64 and 128 CUs 1.6-5.7
// percent faster, whole or spread XCDs), so they are taken whenever six
// loads cover the row.  For 8 KiB rows (11008 x 4096) two-row tiles with x
// once were up to 6.5 percent faster on whole XCDs but up to 7.7 percent
// slower on spread CUs, and stay four-row.  The row shape never changes a
// result: every lane sums its own 16-byte slices in the same order whatever
// the tile.
//
// MFMA tile height by the rows of the busiest CU: 8-row tiles when they cut
// its rows by a fifth or more (fewer tiles than CUs, or a last round that
// 16-row tiles fill unevenly), since a row costs more in an 8-row tile (x is
// read twice as often per W byte); the same bits either way.  Over M =
// 1536..8192 rows of 4096 and 11008, batch 4 and 8, on 64..256 CUs this is
// never more than 5 percent slower than the better height (a rule of one to
// two 16-row tiles per CU was up to 26 percent slower).
static sgdrc_gemv_plan make_plan(uint32_t allowed, int w_dtype, uint32_t M, uint32_t K,
                                 int x_dtype, uint32_t batch)
{
    sgdrc_gemv_plan p{};
    const uint64_t a = allowed ? allowed : 1u;
    const bool mfma = batch >= 3 && w_dtype == x_dtype && w_dtype != SGDRC_F32;
    const uint64_t row_bytes = (uint64_t)K * dtype_size(w_dtype);
    const uint64_t kv = row_bytes / 16u;  // 16-byte slices per row
    if (mfma) {
        const uint64_t r16 = (((M + 15u) / 16u + a - 1u) / a) * 16u;
        const uint64_t r8 = (((M + 7u) / 8u + a - 1u) / a) * 8u;
        p.path = SGDRC_GEMV_MFMA;
        p.rows = 5u * r8 <= 4u * r16 ? 8u : 16u;
        p.loads = (uint32_t)kMfmaSets;
        p.batch_cols = batch <= 4u ? 4u : (uint32_t)kMfmaBatchRows;
        // per output: the MFMAs of one wave in sequence (4 k-steps per
        // 2 KiB chunk, each adding 32 products), then the 8 waves' partials
        const uint64_t chunks = (kv + kMfmaChunkSlices - 1u) / kMfmaChunkSlices;
        p.sum_depth = (uint32_t)(chunks * (uint64_t)kMfmaStepsPerWave + 32u + (kMfmaWaves - 1));
        // x for the whole K staged in LDS once per workgroup at batch 3-4
        // when a row is at most 8 KiB (four rows of x beside the W chunk
        // keep two workgroups per CU): 11008 x 4096 batch 4 2.9-9.7 percent
        // faster on 64..256 CUs (same-box A/B).  Same bits.
        p.x_once = p.batch_cols == 4u && row_bytes <= kXaBytes ? 1u : 0u;
    } else {
        // rows of more than 512 slices of 16 bytes take more than two
        // loads per lane
        const bool long_rows = row_bytes > 512u * 16u;
        // at most six four-row tiles per allowed CU
        const bool few = (M + 3u) / 4u <= 6u * a;
        p.path = SGDRC_GEMV_VALU;
        p.batch_cols = batch <= 1 ? 1u : batch <= 2 ? 2u : batch <= 4 ? 4u : 8u;
        p.rows = 4u;
        p.loads = long_rows && batch <= 2 ? 3u : 2u;
        const bool one_round6 = w_dtype == x_dtype && kv <= 6u * (uint64_t)kGemvThreads;
        if (batch <= 1 && long_rows && (few || one_round6)) {
            p.rows = 2u;
            p.loads = 6u;
        }
        // x once per workgroup when one round of loads covers a row (every
        // tile then reads the same x slices per lane) and x is at least half
        // the bytes a tile reads, batch 1-2 (wider batches would hold too
        // many registers).  Same bits either way.  Measured on MI355X (bf16,
        // 2 MiB pages, eight rotated weight copies, two same-box A/B runs):
        // 4096 x 11008 batch 1 3.1-3.5 percent faster on 256 CUs and
        // 3.6-7.3 percent on 192, 11008 x 4096 batch 2 5.5-9.3 percent
        // faster on 64..256 CUs;
        // with x a quarter of a tile's bytes (four-row tiles, batch 1) it
        // was up to 2.8 percent slower, so those keep per-tile x loads.
        // (W and x of one type, as measured; a wider x would hold twice the
        // registers)
        const uint64_t round_slices = (uint64_t)p.loads * (uint64_t)kGemvThreads;
        p.x_once = w_dtype == x_dtype && kv <= round_slices && p.batch_cols <= 2u &&
                   2u * p.batch_cols >= p.rows ? 1u : 0u;
        // per output: each lane's FMA chain over its slices, the butterfly
        // over 64 lanes, then the 4 waves' partials
        const uint64_t epv = 16u / (uint64_t)dtype_size(w_dtype);
        p.sum_depth = (uint32_t)(((kv + kGemvThreads - 1u) / kGemvThreads) * epv + 6u +
                                 (kGemvWaves - 1));
    }
    p.tiles = (M + p.rows - 1u) / p.rows;
    return p;
}

template <int WT, int XT>
static GemvKernel valu_kernel(const sgdrc_gemv_plan &p)
{
#define SGDRC_VALU(NB, R, U, XO)                                                      \
    if (p.batch_cols == NB && p.rows == R && p.loads == U && p.x_once == (XO ? 1u : 0u)) \
        return k_gemv_valu<WT, XT, NB, R, U, XO>;
    SGDRC_VALU(1, 2, 6, false)
    SGDRC_VALU(1, 4, 3, false)
    SGDRC_VALU(1, 4, 2, false)
    SGDRC_VALU(2, 4, 3, false)
    SGDRC_VALU(2, 4, 2, false)
    SGDRC_VALU(4, 4, 2, false)
    SGDRC_VALU(8, 4, 2, false)
    if constexpr (WT == XT) {  // x once per workgroup: one type only
        SGDRC_VALU(1, 2, 6, true)
        SGDRC_VALU(2, 4, 3, true)
        SGDRC_VALU(2, 4, 2, true)
    }
#undef SGDRC_VALU
    return nullptr;
}

template <int WT>
static GemvKernel valu_kernel_x(int x_dtype, const sgdrc_gemv_plan &p)
{
    switch (x_dtype) {
    case SGDRC_F32: return valu_kernel<WT, SGDRC_F32>(p);
    case SGDRC_BF16: return valu_kernel<WT, SGDRC_BF16>(p);
    default: return valu_kernel<WT, SGDRC_F16>(p);
    }
}

static GemvKernel plan_kernel(const sgdrc_gemv_plan &p, int w_dtype, int x_dtype)
{
    if (p.path == SGDRC_GEMV_MFMA) {
        if (p.batch_cols == 4 && p.x_once) {
            if (p.rows == 16)
                return w_dtype == SGDRC_BF16 ? k_gemm_mfma<SGDRC_BF16, 16, 4, true> : k_gemm_mfma<SGDRC_F16, 16, 4, true>;
            return w_dtype == SGDRC_BF16 ? k_gemm_mfma<SGDRC_BF16, 8, 4, true> : k_gemm_mfma<SGDRC_F16, 8, 4, true>;
        }
        if (p.batch_cols == 4) {
            if (p.rows == 16)
                return w_dtype == SGDRC_BF16 ? k_gemm_mfma<SGDRC_BF16, 16, 4, false> : k_gemm_mfma<SGDRC_F16, 16, 4, false>;
            return w_dtype == SGDRC_BF16 ? k_gemm_mfma<SGDRC_BF16, 8, 4, false> : k_gemm_mfma<SGDRC_F16, 8, 4, false>;
        }
        if (p.rows == 16)
            return w_dtype == SGDRC_BF16 ? k_gemm_mfma<SGDRC_BF16, 16, 8, false> : k_gemm_mfma<SGDRC_F16, 16, 8, false>;
        return w_dtype == SGDRC_BF16 ? k_gemm_mfma<SGDRC_BF16, 8, 8, false> : k_gemm_mfma<SGDRC_F16, 8, 8, false>;
    }
    switch (w_dtype) {
    case SGDRC_F32: return valu_kernel_x<SGDRC_F32>(x_dtype, p);
    case SGDRC_BF16: return valu_kernel_x<SGDRC_BF16>(x_dtype, p);
    default: return valu_kernel_x<SGDRC_F16>(x_dtype, p);
    }
}

static int kernel_occupancy(GemvKernel k, int threads)
{
    static std::mutex mu;
    static std::unordered_map<const void *, int> cache;
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find((const void *)k);
    if (it != cache.end())
        return it->second;
    int n = occupancy(k, threads);
    cache[(const void *)k] = n;
    return n;
}

// Argument checks shared by colored_gemv and colored_gemv_plan.
static int check_gemv_shape(int w_dtype, uint32_t M, uint32_t K, int x_dtype, uint32_t batch)
{
    if (w_dtype < SGDRC_F32 || w_dtype > SGDRC_F16 || x_dtype < SGDRC_F32 || x_dtype > SGDRC_F16)
        return set_error(SGDRC_EINVAL, "unknown dtype (w %d, x %d)", w_dtype, x_dtype);
    if (batch < 1 || batch > SGDRC_MAX_BATCH)
        return set_error(SGDRC_EINVAL, "batch %u outside 1..%d", batch, SGDRC_MAX_BATCH);
    if (M == 0 || K == 0)
        return set_error(SGDRC_EINVAL, "M and K must be positive");
    if (((uint64_t)K * dtype_size(w_dtype)) % 16u)
        return set_error(SGDRC_EINVAL, "K * element size must be a multiple of 16 bytes");
    if ((uint64_t)K * dtype_size(w_dtype) / 16u >= (1ull << 31))
        return set_error(SGDRC_EINVAL, "K too large");
    if ((uint64_t)batch * K * dtype_size(x_dtype) > 0xFFFFFFF0ull)
        return set_error(SGDRC_EINVAL, "x must be smaller than 4 GiB");
    return SGDRC_OK;
}

}  // namespace sgdrc

using namespace sgdrc;

extern "C" {

int colored_gemv_plan(uint32_t allowed_cus, int w_dtype, uint32_t M, uint32_t K, int x_dtype,
                    uint32_t batch, sgdrc_gemv_plan *out)
{
    clear_error();
    if (!out)
        return set_error(SGDRC_EINVAL, "out is NULL");
    if (allowed_cus < 1 || allowed_cus > SGDRC_MAX_CUS)
        return set_error(SGDRC_EINVAL, "allowed_cus %u outside 1..%d", allowed_cus, SGDRC_MAX_CUS);
    int rc = check_gemv_shape(w_dtype, M, K, x_dtype, batch);
    if (rc)
        return rc;
    *out = make_plan(allowed_cus, w_dtype, M, K, x_dtype, batch);
    return SGDRC_OK;
}

int colored_gemv(sgdrc_ctx *ctx, const sgdrc_paged *w, int w_dtype, uint32_t M, uint32_t K,
                 const void *d_x, int x_dtype, uint32_t batch, float *d_y, uint32_t page_shift,
                 void *stream)
{
    clear_error();
    int rc = check_shift(page_shift);
    if (rc)
        return rc;
    if ((rc = check_paged(w, "w")))
        return rc;
    if ((rc = check_gemv_shape(w_dtype, M, K, x_dtype, batch)))
        return rc;
    if (!d_x || !d_y)
        return set_error(SGDRC_EINVAL, "NULL x or y");
    if ((reinterpret_cast<uintptr_t>(d_x) & 15u) || (reinterpret_cast<uintptr_t>(d_y) & 3u))
        return set_error(SGDRC_EINVAL, "x must be 16-byte and y 4-byte aligned");
    {
        // a tile's rows must span at most kPtCap pages (they are staged in LDS)
        const bool mfma = batch >= 3 && w_dtype == x_dtype && w_dtype != SGDRC_F32;
        const uint64_t rows = mfma ? kMfmaRows : kGemvRowsMax;
        const uint64_t span = rows * (uint64_t)K * dtype_size(w_dtype);
        if ((span >> page_shift) + 2 > (uint64_t)kPtCap)
            return set_error(SGDRC_EINVAL, "rows of %llu bytes span too many %u-byte pages",
                             (unsigned long long)((uint64_t)K * dtype_size(w_dtype)),
                             1u << page_shift);
    }
    Ctx *c = nullptr;
    rc = check_ctx(ctx, &c);
    if (rc)
        return rc;

    const sgdrc_gemv_plan plan =
        make_plan((uint32_t)std::max(1, stream_allowed_cus(c, stream)), w_dtype, M, K, x_dtype,
                  batch);
    const GemvKernel k = plan_kernel(plan, w_dtype, x_dtype);
    if (!k)
        return set_error(SGDRC_EINVAL, "no kernel for the plan (library fault)");
    Gate g;
    LaunchInfo li;
    rc = make_gate(c, stream, plan.tiles, kGemvGroupCus, &g, &li, false, true);
    if (rc)
        return rc;
    const int threads = plan.path == SGDRC_GEMV_MFMA ? kMfmaThreads : kGemvThreads;
    const uint32_t grid = gated_grid(c, kernel_occupancy(k, threads), plan.tiles, li);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k, dim3(grid), dim3(threads), 0, s, static_cast<const uint8_t *>(w->pool),
                       w->pt, w->pool_pages, M, K, static_cast<const uint8_t *>(d_x), batch, d_y,
                       page_shift, (uint32_t)plan.tiles, g);
    SGDRC_HIP(hipGetLastError());
    return finish_static_tlog(g, s);
}

}  // extern "C"
