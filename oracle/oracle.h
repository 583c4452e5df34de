/*
 * CPU oracle for the colour-restricted tensor path.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test-suite, the smoke
 * check and the benchmark's CPU-baseline leg may load this library.  It is a
 * plain, slow, single-threaded statement of what each operation computes,
 * written from the definitions; it shares no source, header, table or
 * helper with the HIP library.
 *
 * Every buffer is host memory.  A "pool" is a byte array of whole pages of
 * 2^page_shift bytes; a page table ``pt`` maps logical page j of a tensor to
 * pool page pt[j].
 */
#ifndef SGDRC_ORACLE_H
#define SGDRC_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1, ORACLE_F16 = 2 };

/* Colour of one address under K XOR masks: bit k of the colour is the
 * parity of the AND of the low 48 address bits with mask k.  Written as an
 * explicit loop over address bits.  Linear XOR channel hash of paper
 * section 3.2 (Limitations of GPU Partitioning). */
uint32_t oracle_colour(uint64_t addr, const uint64_t *masks, uint32_t n_masks);

/* The same colour through popcount: bit k = popcount(addr & M_k) mod 2. */
uint32_t oracle_colour_popcount(uint64_t addr, const uint64_t *masks, uint32_t n_masks);

/* colours[i] = colour(addrs[i]); if hist != NULL, hist[c] = number of i with
 * colour c, for c < 2^K (hist is overwritten). */
void oracle_classify(const uint64_t *addrs, uint64_t n, const uint64_t *masks,
                     uint32_t n_masks, uint8_t *colours, uint64_t *hist);

/* Page-table build (paper section 6, SPT steps 1-3): pool page i covers the
 * bytes [a, a + 2^page_shift) with a = origin + i * 2^page_shift; it
 * qualifies when the colour of every one of those bytes is in the 256-bit
 * set ``colour_set``.  Writes the first min(found, n_needed)
 * qualifying page indices in ascending order and returns ``found``, the
 * number of qualifying pages in the whole pool. */
uint64_t oracle_pagetable(const uint64_t *masks, uint32_t n_masks, uint64_t origin,
                          uint32_t page_shift, uint64_t pool_pages,
                          const uint64_t colour_set[4], uint64_t n_needed,
                          uint32_t *pt);

/* Colour through a table of one colour per 2^lut_shift-byte partition
 * (paper section 5.3): entry i covers [origin + i 2^s, origin + (i+1) 2^s).
 * Outside the table, or an entry of 255: no colour, returned as 255. */
uint32_t oracle_lut_colour(uint64_t addr, const uint8_t *lut, uint64_t origin, uint64_t entries,
                           uint32_t lut_shift);

/* colours[i] = oracle_lut_colour(addrs[i]); hist (256 entries, overwritten,
 * may be NULL) counts every colour value including 255. */
void oracle_classify_lut(const uint64_t *addrs, uint64_t n, const uint8_t *lut, uint64_t origin,
                         uint64_t entries, uint32_t lut_shift, uint8_t *colours, uint64_t *hist);

/* Page-table build through a colour table: page i = [addr_origin + i P,
 * + P) qualifies when every partition it touches is in the table and has a
 * colour (not 255) in the set.  As oracle_pagetable otherwise. */
uint64_t oracle_pagetable_lut(const uint8_t *lut, uint64_t origin, uint64_t entries,
                              uint32_t lut_shift, uint64_t addr_origin, uint32_t page_shift,
                              uint64_t pool_pages, const uint64_t colour_set[4],
                              uint64_t n_needed, uint32_t *pt);

/* Bimodal relayout (paper section 7.2): for every logical byte b < n_bytes,
 * dst[pt_dst[b >> s] << s | (b & (2^s - 1))] = src[pt_src[b >> s] << s | ...]. */
void oracle_relayout(uint8_t *dst_pool, const uint32_t *pt_dst, const uint8_t *src_pool,
                     const uint32_t *pt_src, uint64_t n_bytes, uint32_t page_shift);

/* Colour-restricted triad (the re-indexed vector kernel of paper section 6,
 * SPT step 4): a[i] = fmaf(s, c[i], b[i]) for i < n, every element reached
 * through its array's page table. */
void oracle_triad(uint8_t *a_pool, const uint32_t *pt_a, const uint8_t *b_pool,
                  const uint32_t *pt_b, const uint8_t *c_pool, const uint32_t *pt_c,
                  float s, uint64_t n, uint32_t page_shift);

/* Value of one element stored with the given encoding (IEEE binary32,
 * bfloat16 = upper half of a binary32, IEEE binary16). */
double oracle_decode(uint32_t bits, int dtype);

/* GEMV / small-batch GEMM of a memory-bound layer (paper section 7.2):
 * y[b*M + m] = sum_k W[m][k] * x[b][k] in double, W row-major [M x K] read
 * through pt_w, x contiguous [B x K].  If absdot != NULL it receives
 * sum_k |W[m][k] * x[b][k]| (the scale of the rounding-error bound). */
void oracle_gemv(const uint8_t *w_pool, const uint32_t *pt_w, int w_dtype, uint32_t M,
                 uint32_t K, const void *x, int x_dtype, uint32_t B, uint32_t page_shift,
                 double *y, double *absdot);

#ifdef __cplusplus
}
#endif

#endif
