/*
 * CPU oracle for the colour-restricted tensor path -- TEST INFRASTRUCTURE.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg use
 * this file.  Each function is the plain definition of one operation, one
 * element at a time, in the order the definition states; there is no
 * blocking, vectorisation or threading.  Floating-point results that the
 * method leaves to a sum (the GEMV) are accumulated in double.
 *
 * Parity pins (tests/test_oracle_pins.py): every function here is checked
 * against invariants, closed forms, brute force or a library routine that
 * does not call this file.
 */
#include "oracle.h"

#include <math.h>
#include <string.h>

#define ADDR_BITS 48u

/* Paper section 3.2: the XOR channel hash is linear over GF(2); channel bit
 * k is the XOR of the address bits that mask k selects. */
uint32_t oracle_colour(uint64_t addr, const uint64_t *masks, uint32_t n_masks)
{
    uint32_t colour = 0;
    for (uint32_t k = 0; k < n_masks; ++k) {
        uint32_t parity = 0;
        for (uint32_t b = 0; b < ADDR_BITS; ++b) {
            uint32_t abit = (uint32_t)((addr >> b) & 1u);
            uint32_t mbit = (uint32_t)((masks[k] >> b) & 1u);
            parity ^= abit & mbit;
        }
        colour |= parity << k;
    }
    return colour;
}

uint32_t oracle_colour_popcount(uint64_t addr, const uint64_t *masks, uint32_t n_masks)
{
    const uint64_t low48 = (1ull << ADDR_BITS) - 1ull;
    uint32_t colour = 0;
    for (uint32_t k = 0; k < n_masks; ++k) {
        uint32_t ones = (uint32_t)__builtin_popcountll(addr & masks[k] & low48);
        colour |= (ones & 1u) << k;
    }
    return colour;
}

void oracle_classify(const uint64_t *addrs, uint64_t n, const uint64_t *masks,
                     uint32_t n_masks, uint8_t *colours, uint64_t *hist)
{
    if (hist)
        for (uint64_t c = 0; c < (1ull << n_masks); ++c)
            hist[c] = 0;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t c = oracle_colour(addrs[i], masks, n_masks);
        colours[i] = (uint8_t)c;
        if (hist)
            hist[c] += 1;
    }
}

static int in_set(const uint64_t set[4], uint32_t colour)
{
    return (int)((set[colour >> 6] >> (colour & 63u)) & 1u);
}

/* Paper section 6 colours whole sectors: all bytes of a sector lie on the
 * channels of its colour.  A pool page therefore belongs to a colour set
 * only if every byte of it has a colour in the set.  The colour of an
 * address depends only on the address bits that some mask selects, so the
 * colours of the bytes of the page at ``base`` are exactly the colours of
 * base + o for every offset o made of in-page bits that some mask selects
 * (o = 0 among them).  With no mask bit below the page size that is the
 * colour of the page's base alone. */
static int page_in_set(uint64_t base, uint32_t page_shift, const uint64_t *masks,
                       uint32_t n_masks, const uint64_t set[4])
{
    uint64_t selected = 0;
    for (uint32_t k = 0; k < n_masks; ++k)
        selected |= masks[k];
    const uint64_t in_page = selected & ((1ull << page_shift) - 1ull);
    /* o runs over every subset of the bits of in_page, in increasing order:
     * 0, then (o - in_page) & in_page until o == in_page */
    uint64_t o = 0;
    for (;;) {
        if (!in_set(set, oracle_colour(base + o, masks, n_masks)))
            return 0;
        if (o == in_page)
            return 1;
        o = (o - in_page) & in_page;
    }
}

/* Paper section 6, SPT steps 1-3: pages of the reserved pool are sorted
 * into per-colour lists; a tensor takes its pages from the lists of its
 * colours.  Reading used here: ascending pool index, first n pages. */
uint64_t oracle_pagetable(const uint64_t *masks, uint32_t n_masks, uint64_t origin,
                          uint32_t page_shift, uint64_t pool_pages,
                          const uint64_t colour_set[4], uint64_t n_needed,
                          uint32_t *pt)
{
    uint64_t found = 0;
    for (uint64_t i = 0; i < pool_pages; ++i) {
        uint64_t page_addr = origin + (i << page_shift);
        if (page_in_set(page_addr, page_shift, masks, n_masks, colour_set)) {
            if (found < n_needed)
                pt[found] = (uint32_t)i;
            found += 1;
        }
    }
    return found;
}

/* Paper section 5.3: for hashes that are not XOR-linear, a table holds the
 * channel of every partition (1 KiB there).  Entry i is the colour of the
 * bytes [origin + i * 2^s, origin + (i + 1) * 2^s); an address outside the
 * table has no colour, written 255 (as is an entry of 255). */
uint32_t oracle_lut_colour(uint64_t addr, const uint8_t *lut, uint64_t origin, uint64_t entries,
                           uint32_t lut_shift)
{
    if (addr < origin)
        return 255u;
    uint64_t i = (addr - origin) >> lut_shift;
    if (i >= entries)
        return 255u;
    return lut[i];
}

void oracle_classify_lut(const uint64_t *addrs, uint64_t n, const uint8_t *lut, uint64_t origin,
                         uint64_t entries, uint32_t lut_shift, uint8_t *colours, uint64_t *hist)
{
    if (hist)
        for (uint32_t c = 0; c < 256u; ++c)
            hist[c] = 0;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t c = oracle_lut_colour(addrs[i], lut, origin, entries, lut_shift);
        colours[i] = (uint8_t)c;
        if (hist)
            hist[c] += 1;
    }
}

/* Page-table build with a colour table (paper section 6 with the table of
 * section 5.3): pool page i covers the bytes [a, a + 2^page_shift) with
 * a = addr_origin + i * 2^page_shift; it qualifies when every partition it
 * touches lies in the table and has a colour (not 255) in the set.
 * Ascending page order, first n_needed pages; returns all qualifying. */
uint64_t oracle_pagetable_lut(const uint8_t *lut, uint64_t origin, uint64_t entries,
                              uint32_t lut_shift, uint64_t addr_origin, uint32_t page_shift,
                              uint64_t pool_pages, const uint64_t colour_set[4],
                              uint64_t n_needed, uint32_t *pt)
{
    const uint64_t page = 1ull << page_shift;
    const uint64_t part = 1ull << lut_shift;
    uint64_t found = 0;
    for (uint64_t i = 0; i < pool_pages; ++i) {
        const uint64_t first = addr_origin + i * page;
        int ok = 1;
        /* one address per partition the page touches: its first byte, then
         * the start of every later partition inside the page */
        for (uint64_t a = first; a < first + page && ok; a = (a | (part - 1u)) + 1u) {
            uint32_t c = oracle_lut_colour(a, lut, origin, entries, lut_shift);
            ok = c != 255u && in_set(colour_set, c);
        }
        if (ok) {
            if (found < n_needed)
                pt[found] = (uint32_t)i;
            found += 1;
        }
    }
    return found;
}

/* Paper section 7.2: switching a tensor between the all-channel and the
 * restricted page set is a move of its bytes from one set of pages to the
 * other; logical byte b keeps its place in the tensor. */
void oracle_relayout(uint8_t *dst_pool, const uint32_t *pt_dst, const uint8_t *src_pool,
                     const uint32_t *pt_src, uint64_t n_bytes, uint32_t page_shift)
{
    const uint64_t in_page = (1ull << page_shift) - 1ull;
    for (uint64_t b = 0; b < n_bytes; ++b) {
        uint64_t page = b >> page_shift;
        uint64_t off = b & in_page;
        uint64_t d = ((uint64_t)pt_dst[page] << page_shift) + off;
        uint64_t s = ((uint64_t)pt_src[page] << page_shift) + off;
        dst_pool[d] = src_pool[s];
    }
}

/* Address of element i of a float array stored through a page table. */
static uint64_t paged_offset(const uint32_t *pt, uint64_t byte, uint32_t page_shift)
{
    const uint64_t in_page = (1ull << page_shift) - 1ull;
    return ((uint64_t)pt[byte >> page_shift] << page_shift) + (byte & in_page);
}

/* Paper section 6, SPT step 4 (re-indexed vector kernel); a = b + s*c with
 * one rounding (C fmaf). */
void oracle_triad(uint8_t *a_pool, const uint32_t *pt_a, const uint8_t *b_pool,
                  const uint32_t *pt_b, const uint8_t *c_pool, const uint32_t *pt_c,
                  float s, uint64_t n, uint32_t page_shift)
{
    for (uint64_t i = 0; i < n; ++i) {
        uint64_t byte = i * 4u;
        float b, c;
        memcpy(&b, b_pool + paged_offset(pt_b, byte, page_shift), 4);
        memcpy(&c, c_pool + paged_offset(pt_c, byte, page_shift), 4);
        float a = fmaf(s, c, b);
        memcpy(a_pool + paged_offset(pt_a, byte, page_shift), &a, 4);
    }
}

/* IEEE 754 binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits. */
static double decode_f16(uint32_t h)
{
    uint32_t sign = (h >> 15) & 1u;
    uint32_t expo = (h >> 10) & 31u;
    uint32_t frac = h & 1023u;
    double v;
    if (expo == 0)
        v = ldexp((double)frac, -24);               /* zero or subnormal */
    else if (expo == 31)
        v = frac ? NAN : INFINITY;
    else
        v = ldexp((double)(1024u + frac), (int)expo - 25);
    return sign ? -v : v;
}

double oracle_decode(uint32_t bits, int dtype)
{
    float f;
    uint32_t word;
    switch (dtype) {
    case ORACLE_F32:
        word = bits;
        memcpy(&f, &word, 4);
        return (double)f;
    case ORACLE_BF16:
        /* bfloat16 is the upper 16 bits of a binary32 */
        word = (bits & 0xFFFFu) << 16;
        memcpy(&f, &word, 4);
        return (double)f;
    case ORACLE_F16:
        return decode_f16(bits & 0xFFFFu);
    default:
        return NAN;
    }
}

static uint32_t elem_size(int dtype)
{
    return dtype == ORACLE_F32 ? 4u : 2u;
}

static uint32_t load_bits(const uint8_t *p, uint32_t size)
{
    uint32_t v = 0;
    memcpy(&v, p, size);  /* little-endian host */
    return v;
}

/* Memory-bound layer of paper section 7.2: a plain dot product per output,
 * W element (m, k) found through the page table at logical byte
 * (m*K + k) * element size. */
void oracle_gemv(const uint8_t *w_pool, const uint32_t *pt_w, int w_dtype, uint32_t M,
                 uint32_t K, const void *x, int x_dtype, uint32_t B, uint32_t page_shift,
                 double *y, double *absdot)
{
    const uint32_t wsz = elem_size(w_dtype), xsz = elem_size(x_dtype);
    const uint8_t *xb = (const uint8_t *)x;
    for (uint32_t b = 0; b < B; ++b) {
        for (uint32_t m = 0; m < M; ++m) {
            double acc = 0.0, mag = 0.0;
            for (uint32_t k = 0; k < K; ++k) {
                uint64_t byte = ((uint64_t)m * K + k) * wsz;
                double w = oracle_decode(load_bits(w_pool + paged_offset(pt_w, byte, page_shift), wsz), w_dtype);
                double xv = oracle_decode(load_bits(xb + ((uint64_t)b * K + k) * xsz, xsz), x_dtype);
                acc += w * xv;
                mag += fabs(w * xv);
            }
            y[(uint64_t)b * M + m] = acc;
            if (absdot)
                absdot[(uint64_t)b * M + m] = mag;
        }
    }
}
