// Contiguous, ungated counterparts of the library's paged kernels: the same
// per-lane work (tile shape, loads in flight, arithmetic) on plain arrays,
// without page tables, CU gate or tile queues.  Only compiled, never
// launched: tests/resource_report.py compares their register and LDS use
// with the library's kernels (the analogue of counting the registers that
// re-indexing adds to a kernel, paper section 9.1.2).
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// triad a = fmaf(s, c, b): U 16-byte slices per lane and array in flight
template <int U>
__global__ __launch_bounds__(256) void plain_triad(u32x4 *__restrict__ a, const u32x4 *__restrict__ b,
                                                   const u32x4 *__restrict__ c, float s, uint64_t nv)
{
    for (uint64_t base = (uint64_t)blockIdx.x * 256u * U + threadIdx.x; base < nv;
         base += (uint64_t)gridDim.x * 256u * U) {
        u32x4 vb[U], vc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i = base + (uint64_t)u * 256u;
            vb[u] = i < nv ? __builtin_nontemporal_load(b + i) : u32x4{0, 0, 0, 0};
            vc[u] = i < nv ? __builtin_nontemporal_load(c + i) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i = base + (uint64_t)u * 256u;
            u32x4 r;
            r.x = __float_as_uint(__builtin_fmaf(s, __uint_as_float(vc[u].x), __uint_as_float(vb[u].x)));
            r.y = __float_as_uint(__builtin_fmaf(s, __uint_as_float(vc[u].y), __uint_as_float(vb[u].y)));
            r.z = __float_as_uint(__builtin_fmaf(s, __uint_as_float(vc[u].z), __uint_as_float(vb[u].z)));
            r.w = __float_as_uint(__builtin_fmaf(s, __uint_as_float(vc[u].w), __uint_as_float(vb[u].w)));
            if (i < nv)
                __builtin_nontemporal_store(r, a + i);
        }
    }
}

// copy (the relayout with identity tables): U slices per lane in flight
template <int U>
__global__ __launch_bounds__(256) void plain_copy(u32x4 *__restrict__ d, const u32x4 *__restrict__ s, uint64_t nv)
{
    for (uint64_t base = (uint64_t)blockIdx.x * 256u * U + threadIdx.x; base < nv;
         base += (uint64_t)gridDim.x * 256u * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i = base + (uint64_t)u * 256u;
            v[u] = i < nv ? __builtin_nontemporal_load(s + i) : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i = base + (uint64_t)u * 256u;
            if (i < nv)
                __builtin_nontemporal_store(v[u], d + i);
        }
    }
}

// batch-1 bf16 GEMV, R rows per workgroup, U slices per lane and row, the
// library's lane layout and fixed-order reductions
template <int R, int U>
__global__ __launch_bounds__(256) void plain_gemv(const u32x4 *__restrict__ W, const u32x4 *__restrict__ x,
                                                  float *__restrict__ y, uint32_t M, uint32_t K)
{
    __shared__ float s_red[4][R];
    const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63u;
    const uint32_t KV = K / 8u, m0 = blockIdx.x * R;
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        acc[r] = 0.f;
    for (uint32_t j = 0; (j * 4u + wave) * 64u < KV; j += U) {
        u32x4 wv[U][R], xv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t kv = ((j + u) * 4u + wave) * 64u + lane;
            const bool ok = kv < KV;
            xv[u] = ok ? x[kv] : u32x4{0, 0, 0, 0};
#pragma unroll
            for (int r = 0; r < R; ++r)
                wv[u][r] = ok && m0 + r < M ? __builtin_nontemporal_load(W + (uint64_t)(m0 + r) * KV + kv)
                                            : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const u32x4 w = wv[u][r], xx = xv[u];
                const uint32_t ws[4] = {w.x, w.y, w.z, w.w}, xs[4] = {xx.x, xx.y, xx.z, xx.w};
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc[r] = __builtin_fmaf(__uint_as_float(ws[q] << 16), __uint_as_float(xs[q] << 16), acc[r]);
                    acc[r] = __builtin_fmaf(__uint_as_float(ws[q] & 0xFFFF0000u),
                                            __uint_as_float(xs[q] & 0xFFFF0000u), acc[r]);
                }
            }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        float v = acc[r];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
            v += __shfl_xor(v, off, 64);
        acc[r] = v;
    }
    if (lane == 0)
#pragma unroll
        for (int r = 0; r < R; ++r)
            s_red[wave][r] = acc[r];
    __syncthreads();
    if (threadIdx.x < (uint32_t)R && m0 + threadIdx.x < M)
        y[m0 + threadIdx.x] = s_red[0][threadIdx.x] + s_red[1][threadIdx.x] + s_red[2][threadIdx.x] +
                              s_red[3][threadIdx.x];
}

// classify: each wavefront L 16-byte loads per lane (2 addresses each), six
// byte-table lookups per address from LDS, colours re-packed through LDS
template <int L>
__global__ __launch_bounds__(256) void plain_classify(const u32x4 *__restrict__ addrs, uint32_t n_tiles,
                                                      const uint8_t *__restrict__ tables,
                                                      u32x4 *__restrict__ colours)
{
    __shared__ __attribute__((aligned(16))) uint16_t s_col[4][64 * L];
    __shared__ uint8_t t[6][256];
    for (uint32_t i = threadIdx.x; i < 6u * 256u; i += 256u)
        t[i >> 8][i & 255u] = tables[i];
    __syncthreads();
    const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63u;
    for (uint32_t tile = blockIdx.x * 4u + wave; tile < n_tiles; tile += gridDim.x * 4u) {
        u32x4 v[L];
#pragma unroll
        for (int j = 0; j < L; ++j)
            v[j] = __builtin_nontemporal_load(addrs + (uint64_t)tile * 64u * L + j * 64u + lane);
#pragma unroll
        for (int j = 0; j < L; ++j) {
            const uint32_t c0 = t[0][v[j].x & 255u] ^ t[1][(v[j].x >> 8) & 255u] ^ t[2][(v[j].x >> 16) & 255u] ^
                                t[3][v[j].x >> 24] ^ t[4][v[j].y & 255u] ^ t[5][(v[j].y >> 8) & 255u];
            const uint32_t c1 = t[0][v[j].z & 255u] ^ t[1][(v[j].z >> 8) & 255u] ^ t[2][(v[j].z >> 16) & 255u] ^
                                t[3][v[j].z >> 24] ^ t[4][v[j].w & 255u] ^ t[5][(v[j].w >> 8) & 255u];
            s_col[wave][j * 64u + lane] = (uint16_t)(c0 | (c1 << 8));
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < L / 8; ++q)
            __builtin_nontemporal_store(*reinterpret_cast<const u32x4 *>(&s_col[wave][q * 512u + lane * 8u]),
                                        colours + (uint64_t)tile * 4u * L + q * 64u + lane);
        __builtin_amdgcn_wave_barrier();
    }
}

template __global__ void plain_triad<16>(u32x4 *, const u32x4 *, const u32x4 *, float, uint64_t);
template __global__ void plain_copy<16>(u32x4 *, const u32x4 *, uint64_t);
template __global__ void plain_gemv<2, 6>(const u32x4 *, const u32x4 *, float *, uint32_t, uint32_t);
template __global__ void plain_gemv<4, 3>(const u32x4 *, const u32x4 *, float *, uint32_t, uint32_t);
template __global__ void plain_gemv<4, 2>(const u32x4 *, const u32x4 *, float *, uint32_t, uint32_t);
template __global__ void plain_classify<8>(const u32x4 *, uint32_t, const uint8_t *, u32x4 *);
