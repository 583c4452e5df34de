"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test ties one oracle function to an invariant, a closed form, brute
force on a tiny input, or a library routine (numpy, Python's exact
rationals).  A plausible slip in the oracle -- a dropped address word, a
reversed colour bit order, a wrong page index, a transposed GEMV operand,
a double rounding in the triad -- fails at least one of them.
"""
from fractions import Fraction
import itertools

import numpy as np
import pytest

import synth

def parity(v: int) -> int:
    return bin(v).count("1") & 1


# ---------------------------------------------------------------- colour ---

def test_colour_hand_worked_example(orc):
    # masks: M0 selects bits 9 and 11, M1 selects bits 9 and 10
    masks = [(1 << 9) | (1 << 11), (1 << 9) | (1 << 10)]
    assert orc.colour(0, masks) == 0
    assert orc.colour(1 << 9, masks) == 0b11     # both masks see one set bit
    assert orc.colour(1 << 10, masks) == 0b10    # only M1
    assert orc.colour(1 << 11, masks) == 0b01    # only M0
    assert orc.colour((1 << 9) | (1 << 10) | (1 << 11), masks) == 0b00
    assert orc.colour((1 << 12) | (1 << 8), masks) == 0  # unselected bits


def test_colour_bitloop_matches_popcount_form(orc):
    masks = synth.xor_masks(6, seed=3)
    addrs = synth.page_addresses(2000, seed=5, page_bits=8)
    for a in addrs[:2000]:
        assert orc.colour(int(a), masks) == orc.colour_popcount(int(a), masks)


def test_colour_is_gf2_linear(orc):
    masks = synth.xor_masks(5, seed=7)
    assert orc.colour(0, masks) == 0
    a = synth.page_addresses(500, seed=11, page_bits=0)
    b = synth.page_addresses(500, seed=12, page_bits=0)
    for x, y in zip(a, b):
        x, y = int(x), int(y)
        assert orc.colour(x ^ y, masks) == orc.colour(x, masks) ^ orc.colour(y, masks)


@pytest.mark.parametrize("base_bit", [0, 16, 32, 44])
def test_single_bit_masks_extract_address_bits(orc, base_bit):
    k = 4
    masks = [1 << (base_bit + j) for j in range(k)]
    for a in synth.page_addresses(300, seed=base_bit, page_bits=0):
        a = int(a)
        assert orc.colour(a, masks) == (a >> base_bit) & 0xF


def test_bits_at_and_above_48_are_inert(orc):
    masks = [(1 << 47) | (1 << 20), (1 << 40) | (1 << 3)]
    assert orc.colour(1 << 47, masks) == 0b01
    for a in synth.page_addresses(200, seed=2, page_bits=0):
        a = int(a)
        assert orc.colour(a | (0xFFFF << 48), masks) == orc.colour(a, masks)


def test_range_mask_is_parity_of_the_range(orc):
    # one mask covering bits 8..40: colour = parity of those address bits
    full = ((1 << 33) - 1) << 8
    for a in synth.page_addresses(300, seed=9, page_bits=0):
        a = int(a)
        assert orc.colour(a, [full]) == parity(a & full)


def test_equal_class_sizes_over_full_rank_bit_subset(orc):
    # enumerate every combination of 10 address bits; masks restricted to
    # those bits have rank K = 4, so each of the 16 colours appears 2^(10-4)
    bits = [12, 13, 15, 17, 20, 22, 25, 31, 36, 40]
    masks = synth.xor_masks(4, seed=21, min_bit=12)
    sub = [sum(((m >> b) & 1) << i for i, b in enumerate(bits)) for m in masks]
    assert synth.gf2_rank(sub) == 4
    counts = np.zeros(16, dtype=np.int64)
    for combo in range(1 << len(bits)):
        a = sum(((combo >> i) & 1) << b for i, b in enumerate(bits))
        counts[orc.colour(a, masks)] += 1
    assert (counts == 64).all()


# -------------------------------------------------------------- classify ---

def test_classify_partitions_indices_and_counts_duplicates(orc):
    masks = synth.xor_masks(4, seed=1, min_bit=16)
    addrs = synth.page_addresses(4096, seed=0)
    addrs[100:110] = addrs[5]          # duplicates are classified independently
    colours, hist = orc.classify(addrs, masks)
    assert colours.dtype == np.uint8 and colours.size == addrs.size
    assert int(hist.sum()) == addrs.size
    assert (hist == np.bincount(colours, minlength=16)).all()
    assert (colours[100:110] == colours[5]).all()
    for i in range(0, addrs.size, 37):
        assert colours[i] == orc.colour_popcount(int(addrs[i]), masks)


def test_classify_empty(orc):
    colours, hist = orc.classify(np.zeros(0, dtype=np.uint64), [1 << 12])
    assert colours.size == 0 and (hist == 0).all()


# ------------------------------------------------------------ page table ---

def _page_colour_py(masks, addr):
    return sum(parity(addr & m) << k for k, m in enumerate(masks))


@pytest.mark.parametrize("shift", [12, 16, 21])
def test_pagetable_invariants(orc, shift):
    masks = synth.xor_masks(4, seed=1, min_bit=shift)
    origin = 1 << 40
    pool_pages = 700
    S = [0, 1, 2, 3]
    words = synth.colour_set_bits(S)
    n = 30
    pt, found = orc.pagetable(masks, origin, shift, pool_pages, words, n)
    assert pt.size == n
    assert (np.diff(pt.astype(np.int64)) > 0).all()
    for j, p in enumerate(pt):
        assert _page_colour_py(masks, origin + (int(p) << shift)) in S
    chosen = set(int(p) for p in pt)
    for i in range(int(pt[-1])):
        if i not in chosen:
            assert _page_colour_py(masks, origin + (i << shift)) not in S
    # count = sum over S of the pool's colour histogram
    page_addrs = np.array([origin + (i << shift) for i in range(pool_pages)], dtype=np.uint64)
    _, hist = orc.classify(page_addrs, masks)
    assert found == int(sum(hist[c] for c in S))


def test_pagetable_isolation_and_partition(orc):
    shift = 16
    masks = synth.xor_masks(3, seed=4, min_bit=shift)
    pool = 512
    seen = np.zeros(pool, dtype=np.int64)
    for c in range(8):
        pt, found = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits([c]), pool)
        assert pt.size == found
        seen[pt] += 1
    assert (seen == 1).all()           # singleton sets partition the pool
    a, _ = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits([0, 1, 2]), pool)
    b, _ = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits([3, 4, 5, 6, 7]), pool)
    assert not set(a.tolist()) & set(b.tolist())   # disjoint colours, disjoint pages


def test_pagetable_single_bit_masks_closed_form(orc):
    shift = 16
    masks = [1 << (shift + k) for k in range(3)]   # page i has colour i mod 8
    pt, found = orc.pagetable(masks, 0, shift, 100, synth.colour_set_bits([5]), 7)
    assert found == len(range(5, 100, 8))
    assert pt.tolist() == list(range(5, 100, 8))[:7]


def test_pagetable_shortfall_returns_every_qualifying_page(orc):
    masks = [1 << 16, 1 << 17]
    pt, found = orc.pagetable(masks, 0, 16, 10, synth.colour_set_bits([3]), 50)
    assert found == 2 and pt.tolist() == [3, 7]


# -------------------------------------------------------------- relayout ---

def _pool_view(pool, shift):
    return pool.reshape(-1, 1 << shift)


@pytest.mark.parametrize("n_bytes", [3 * 4096, 3 * 4096 - 1, 5 * 4096 + 17, 1])
def test_relayout_identity_tables_are_memcpy(orc, n_bytes):
    shift = 12
    pages = -(-n_bytes // 4096)
    src = synth.random_bytes(8 * 4096, seed=1)
    dst = np.full(8 * 4096, 0xA5, dtype=np.uint8)
    ident = np.arange(pages, dtype=np.uint32)
    orc.relayout(dst, ident, src, ident, n_bytes, shift)
    assert (dst[:n_bytes] == src[:n_bytes]).all()
    assert (dst[n_bytes:] == 0xA5).all()   # tail of the last page untouched


def test_relayout_matches_numpy_page_gather(orc):
    shift = 12
    pages = 20
    src = synth.random_bytes(64 * 4096, seed=2)
    dst = np.zeros(48 * 4096, dtype=np.uint8)
    pt_s = synth.random_permutation(64, seed=3)[:pages]
    pt_d = synth.random_permutation(48, seed=4)[:pages]
    orc.relayout(dst, pt_d, src, pt_s, pages * 4096, shift)
    expect = np.zeros_like(dst)
    _pool_view(expect, shift)[pt_d.astype(np.int64)] = _pool_view(src, shift)[pt_s.astype(np.int64)]
    assert (dst == expect).all()


def test_relayout_round_trip_is_identity_and_keeps_nan_payloads(orc):
    shift = 16
    masks = synth.xor_masks(6, seed=1, min_bit=shift)
    n_pages = 24
    data = synth.random_u16(n_pages << (shift - 1), seed=5)     # fp16 bit patterns
    all_pt = np.arange(n_pages, dtype=np.uint32)
    s_pt, found = orc.pagetable(masks, 0, shift, 4 * n_pages * 4, synth.colour_set_bits(range(16)),
                                n_pages)
    assert found >= n_pages
    restricted = np.zeros((4 * n_pages * 4) << (shift - 1), dtype=np.uint16)
    back = np.zeros_like(data)
    orc.relayout(restricted, s_pt, data, all_pt, data.nbytes, shift)
    orc.relayout(back, all_pt, restricted, s_pt, data.nbytes, shift)
    assert (back.view(np.uint16) == data.view(np.uint16)).all()
    nan_mask = np.isnan(data.view(np.float16))
    assert nan_mask.any()


# ----------------------------------------------------------------- triad ---

def _nearest_f32(q: Fraction) -> np.float32:
    """Round an exact rational to float32, ties to even, by exact comparison."""
    f = np.float32(float(q))
    best = None
    for cand in (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))):
        err = abs(Fraction(float(cand)) - q)
        key = (err, int(cand.view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, cand)
    return best[1]


def test_triad_identity_pages_equals_exact_sum_rounded_once(orc):
    # U[-1,1) values are multiples of 2^-23 and |s*c + b| < 4, so s*c + b is
    # exact in float64 and one conversion to float32 is the single rounding
    shift = 12
    n = 5 * 1024 + 77
    pages = -(-n * 4 // 4096)
    b = np.zeros(pages * 1024, dtype=np.float32)
    c = np.zeros_like(b)
    b[:n] = synth.uniform_f32(n, seed=1)
    c[:n] = synth.uniform_f32(n, seed=2)
    a = np.full_like(b, np.float32(7.0))
    ident = np.arange(pages, dtype=np.uint32)
    orc.triad(a, ident, b, ident, c, ident, 3.0, n, shift)
    expect = (np.float64(3.0) * c[:n].astype(np.float64) + b[:n].astype(np.float64)).astype(np.float32)
    assert (a[:n].view(np.uint32) == expect.view(np.uint32)).all()
    assert (a[n:] == np.float32(7.0)).all()


def test_triad_single_rounding_against_exact_rationals(orc):
    rng = np.random.default_rng(8)
    n = 1500
    # full-range magnitudes, where a double-rounded s*c + b would differ
    b = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    c = (rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32)
    s = np.float32(1.0000001)
    ident = np.arange(2, dtype=np.uint32)
    bp = np.zeros(2048, dtype=np.float32); bp[:n] = b
    cp = np.zeros(2048, dtype=np.float32); cp[:n] = c
    ap = np.zeros(2048, dtype=np.float32)
    orc.triad(ap, ident, bp, ident, cp, ident, float(s), n, 12)
    for i in range(n):
        exact = Fraction(float(s)) * Fraction(float(c[i])) + Fraction(float(b[i]))
        assert ap[i].view(np.uint32) == _nearest_f32(exact).view(np.uint32), i


def test_triad_special_cases_and_paging(orc):
    shift = 12
    n = 3 * 1024
    b = synth.uniform_f32(n, seed=3)
    c = synth.uniform_f32(n, seed=4)
    ident = np.arange(3, dtype=np.uint32)
    a = np.zeros(n, dtype=np.float32)
    orc.triad(a, ident, b, ident, c, ident, 0.0, n, shift)
    assert (a == b).all()
    orc.triad(a, ident, b, ident, np.zeros_like(c), ident, 3.0, n, shift)
    assert (a == b).all()
    # paged: scatter b and c over shuffled pool pages, result lands on pt_a
    contiguous = np.zeros(n, dtype=np.float32)
    orc.triad(contiguous, ident, b, ident, c, ident, 3.0, n, shift)
    pt_b = synth.random_permutation(8, seed=1)[:3]
    pt_c = synth.random_permutation(8, seed=2)[:3]
    pt_a = synth.random_permutation(8, seed=3)[:3]
    bp = np.zeros(8 * 1024, dtype=np.float32); cp = np.zeros_like(bp); ap = np.zeros_like(bp)
    bp.reshape(8, 1024)[pt_b.astype(np.int64)] = b.reshape(3, 1024)
    cp.reshape(8, 1024)[pt_c.astype(np.int64)] = c.reshape(3, 1024)
    orc.triad(ap, pt_a, bp, pt_b, cp, pt_c, 3.0, n, shift)
    got = ap.reshape(8, 1024)[pt_a.astype(np.int64)].reshape(-1)
    assert (got.view(np.uint32) == contiguous.view(np.uint32)).all()


# ---------------------------------------------------------------- decode ---

def test_decode_f16_all_patterns_match_numpy(orc):
    pats = np.arange(1 << 16, dtype=np.uint32)
    ref = pats.astype(np.uint16).view(np.float16).astype(np.float64)
    got = np.array([orc.decode(int(p), orc.F16) for p in pats])
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all()
    assert np.signbit(got[0x8000]) and got[0x8000] == 0.0


def test_decode_bf16_and_f32_match_numpy_views(orc):
    pats = synth.random_u16(3000, seed=1).astype(np.uint32)
    with np.errstate(invalid="ignore"):
        ref = (pats << np.uint32(16)).view(np.float32).astype(np.float64)
    got = np.array([orc.decode(int(p), orc.BF16) for p in pats])
    assert ((got == ref) | (np.isnan(got) & np.isnan(ref))).all()
    f = synth.normal_f32(500, seed=2)
    got = np.array([orc.decode(int(u), orc.F32) for u in f.view(np.uint32)])
    assert (got == f.astype(np.float64)).all()


def test_bf16_rounding_helper_is_nearest_even():
    # the input generator's float32 -> bf16 rounding, checked on exact cases
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9], dtype=np.float32)
    bits = synth.f32_to_bf16_bits(vals)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    assert back.tolist() == [1.0, 1.0, 1.0 + 2 ** -6, 1.0]


# ------------------------------------------------------------------ GEMV ---

def _decode_np(bits, dtype, orc):
    if dtype == orc.F32:
        return bits.view(np.float32).astype(np.float64)
    if dtype == orc.BF16:
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return bits.view(np.float16).astype(np.float64)


def test_gemv_contiguous_fp32_matches_numpy_matmul(orc):
    M, K, B = 37, 1000, 3           # rows of 4000 B straddle 4 KiB pages
    shift = 12
    w = synth.normal_f32(M * K, seed=1)
    x = synth.normal_f32(B * K, seed=2)
    pages = -(-w.nbytes // 4096)
    pool = np.zeros(pages * 1024, dtype=np.float32); pool[:w.size] = w
    y, ad = orc.gemv(pool, np.arange(pages, dtype=np.uint32), orc.F32, M, K, x, orc.F32, B, shift)
    W = w.reshape(M, K).astype(np.float64)
    X = x.reshape(B, K).astype(np.float64)
    ref = X @ W.T
    assert y.shape == (B, M)
    assert np.all(np.abs(y - ref) <= 1e-12 * (np.abs(X) @ np.abs(W).T))
    assert np.allclose(ad, np.abs(X) @ np.abs(W).T, rtol=1e-12)


@pytest.mark.parametrize("wd,xd", [(1, 1), (2, 2), (1, 0), (0, 1)])
def test_gemv_paged_mixed_dtypes_match_numpy_gather(orc, wd, xd):
    M, K, B = 24, 640, 2
    shift = 12
    wsz = 4 if wd == orc.F32 else 2
    xsz = 4 if xd == orc.F32 else 2
    rng = np.random.default_rng(5)
    if wd == orc.F32:
        wbits = synth.normal_f32(M * K, seed=3).view(np.uint32)
    elif wd == orc.BF16:
        wbits = synth.normal_bf16(M * K, seed=3, sigma=0.02)
    else:
        wbits = synth.normal_f32(M * K, seed=3).astype(np.float16).view(np.uint16)
    if xd == orc.F32:
        xbits = synth.normal_f32(B * K, seed=4).view(np.uint32)
    elif xd == orc.BF16:
        xbits = synth.normal_bf16(B * K, seed=4)
    else:
        xbits = synth.normal_f32(B * K, seed=4).astype(np.float16).view(np.uint16)
    wbytes = wbits.view(np.uint8)
    pages = -(-wbytes.size // 4096)
    pool_pages = pages + 9
    pt = rng.permutation(pool_pages)[:pages].astype(np.uint32)
    padded = np.zeros(pages * 4096, dtype=np.uint8); padded[:wbytes.size] = wbytes
    pool = np.zeros(pool_pages * 4096, dtype=np.uint8)
    pool.reshape(pool_pages, 4096)[pt.astype(np.int64)] = padded.reshape(pages, 4096)
    y, _ = orc.gemv(pool, pt, wd, M, K, xbits, xd, B, shift)
    W = _decode_np(wbits, wd, orc).reshape(M, K)
    X = _decode_np(xbits, xd, orc).reshape(B, K)
    ref = X @ W.T
    assert np.all(np.abs(y - ref) <= 1e-12 * (np.abs(X) @ np.abs(W).T) + 1e-300)
    del wsz, xsz


def test_gemv_closed_forms(orc):
    K = 256
    ident = np.eye(K, dtype=np.float32).reshape(-1)
    pt = np.arange(K * K * 4 // 4096, dtype=np.uint32)
    x = synth.normal_f32(2 * K, seed=6)
    y, _ = orc.gemv(ident, pt, orc.F32, K, K, x, orc.F32, 2, 12)
    assert (y == x.reshape(2, K).astype(np.float64)).all()
    ones = np.ones(K * K, dtype=np.float32)
    y, _ = orc.gemv(ones, pt, orc.F32, K, K, np.ones(K, dtype=np.float32), orc.F32, 1, 12)
    assert (y == K).all()
    # W with one non-zero column j picks x[:, j] for every row: catches W^T
    M = 64
    w = np.zeros((M, K), dtype=np.float32); w[:, 5] = np.arange(M, dtype=np.float32)
    y, _ = orc.gemv(w.reshape(-1), np.arange(M * K * 4 // 4096, dtype=np.uint32), orc.F32, M, K,
                    x, orc.F32, 2, 12)
    assert (y == np.outer(x.reshape(2, K)[:, 5], np.arange(M))).all()


def test_gemv_tiny_exact_rational_sum(orc):
    M, K, B = 3, 50, 2
    w = synth.normal_f32(1024, seed=7)        # one 4 KiB page
    x = synth.normal_f32(B * K, seed=8)
    y, _ = orc.gemv(w, np.zeros(1, dtype=np.uint32), orc.F32, M, K, x, orc.F32, B, 12)
    for b, m in itertools.product(range(B), range(M)):
        exact = sum(Fraction(float(w[m * K + k])) * Fraction(float(x[b * K + k])) for k in range(K))
        assert abs(Fraction(y[b, m]) - exact) <= Fraction(K * 2 ** -52) * sum(
            abs(Fraction(float(w[m * K + k])) * Fraction(float(x[b * K + k]))) for k in range(K))


# ------------------------------------------------ colour table (section 5.3)
# The table form of the hash: one colour per 2^s-byte partition.

def test_lut_colour_hand_worked(orc):
    lut = np.array([3, 1, 255, 0], dtype=np.uint8)     # partitions of 1 KiB from 4096
    assert orc.lut_colour(4096, lut, 4096, 10) == 3
    assert orc.lut_colour(4096 + 1500, lut, 4096, 10) == 1
    assert orc.lut_colour(4096 + 2048 + 5, lut, 4096, 10) == 255   # entry 255: no colour
    assert orc.lut_colour(4096 + 3 * 1024 + 1023, lut, 4096, 10) == 0
    assert orc.lut_colour(4095, lut, 4096, 10) == 255              # below the table
    assert orc.lut_colour(4096 + 4 * 1024, lut, 4096, 10) == 255   # past its end
    addrs = np.array([4096, 4096 + 1500, 4095, 4096 + 3100, 4096 + 1024], dtype=np.uint64)
    col, hist = orc.classify_lut(addrs, lut, 4096, 10)
    assert col.tolist() == [3, 1, 255, 0, 1]
    assert hist[1] == 2 and hist[3] == 1 and hist[0] == 1 and hist[255] == 1 and hist.sum() == 5


def test_pagetable_lut_hand_worked(orc):
    lut = np.array([3, 1, 255, 0], dtype=np.uint8)
    S = synth.colour_set_bits([0, 1, 3])
    # 2 KiB pages from 4096: [p0 p1] = (3, 1) ok; [p2 p3] = (255, 0) no; past the table no
    pt, found = orc.pagetable_lut(lut, 4096, 10, 4096, 11, 3, S, 3)
    assert found == 1 and pt.tolist() == [0]
    # 512 B pages from 4608: one partition each -> colours 3, 1, 1, 255, 255, 0, 0, (past)
    pt, found = orc.pagetable_lut(lut, 4096, 10, 4608, 9, 8, synth.colour_set_bits([1]), 8)
    assert found == 2 and pt.tolist() == [1, 2]
    pt, found = orc.pagetable_lut(lut, 4096, 10, 4608, 9, 8, synth.colour_set_bits([0, 3]), 8)
    assert pt.tolist() == [0, 5, 6] and found == 3


def test_lut_from_xor_hash_agrees_with_the_xor_path(orc):
    """A table filled with the XOR colours of the partition bases gives the
    XOR results: classify for masks above the partition bits, and the page
    table for masks above the page bits (colour constant over a page)."""
    s, origin = 10, 1 << 30
    entries = 1 << 14
    masks = [m & ~((1 << 14) - 1) for m in synth.xor_masks(5, seed=4, min_bit=14)]
    lut = np.array([orc.colour(origin + (i << s), masks) for i in range(entries)], dtype=np.uint8)
    rng = np.random.default_rng(5)
    addrs = (origin + rng.integers(0, entries << s, size=5000)).astype(np.uint64)
    got, gh = orc.classify_lut(addrs, lut, origin, s)
    ref, rh = orc.classify(addrs, masks)
    assert (got == ref).all() and (gh[:32] == rh).all() and gh[32:].sum() == 0
    S = synth.colour_set_bits([1, 4, 9, 30])
    for shift in (13, 14):
        pages = (entries << s) >> shift
        got_pt, gf = orc.pagetable_lut(lut, origin, s, origin, shift, pages, S, pages)
        ref_pt, rf = orc.pagetable(masks, origin, shift, pages, S, pages)
        assert gf == rf and (got_pt == ref_pt).all()


def test_pagetable_lut_needs_every_partition_of_the_page(orc):
    """Masks below the page bits make partitions of one page differ; a page
    then qualifies only if all of them are in the set, so the table form
    takes a subset of the pages the base-address rule takes.  The XOR path
    applies the same whole-page rule by enumerating in-page mask bits, so
    the two forms give the same table whenever no mask bit lies below the
    partition size."""
    s, origin = 10, 0
    entries = 1 << 12
    masks = [m & ~((1 << 10) - 1) for m in synth.xor_masks(4, seed=6, min_bit=10)]
    lut = np.array([orc.colour(origin + (i << s), masks) for i in range(entries)], dtype=np.uint8)
    S = synth.colour_set_bits(range(10))
    shift = 12
    pages = (entries << s) >> shift
    got_pt, gf = orc.pagetable_lut(lut, origin, s, origin, shift, pages, S, pages)
    base = [i for i in range(pages) if _page_colour_py(masks, origin + (i << shift)) < 10]
    assert set(got_pt.tolist()) < set(base)
    for p in got_pt:
        cols = [orc.colour((int(p) << shift) + (j << s), masks) for j in range(4)]
        assert all(c < 10 for c in cols)
    xor_pt, xf = orc.pagetable(masks, origin, shift, pages, S, pages)
    assert xf == gf and (xor_pt == got_pt).all()


# --------------------------------------------- whole pages (paper section 6) ---

def _np_colours(addrs, masks):
    """Colours of many addresses by numpy bit counting (independent of the C
    oracle): bit k = parity of the bits of addr & M_k."""
    a = np.asarray(addrs, dtype=np.uint64)
    out = np.zeros(a.shape, dtype=np.int64)
    for k, m in enumerate(masks):
        v = a & np.uint64(m)
        par = np.zeros(a.shape, dtype=np.uint64)
        for b in range(48):
            par ^= (v >> np.uint64(b)) & np.uint64(1)
        out |= par.astype(np.int64) << k
    return out


@pytest.mark.parametrize("shift,lo,seed", [(10, 8, 3), (11, 9, 4), (12, 10, 5)])
def test_pagetable_whole_page_rule_brute_force(orc, shift, lo, seed):
    """Masks that reach below the page size: a page qualifies exactly when
    the colour of every one of its bytes is in the set (brute force over all
    bytes of every page)."""
    masks = synth.xor_masks(3, seed=seed, min_bit=lo, hi_bit=lo + 12)
    origin = 7 << 30
    pool = 96
    P = 1 << shift
    addrs = origin + np.arange(pool * P, dtype=np.uint64)
    cols = _np_colours(addrs, masks).reshape(pool, P)
    for S in ([0, 1, 2, 3], [0, 2, 4, 6], [1, 3, 5, 7], [0, 1, 4, 5, 6, 7], list(range(8)), [5]):
        member = np.isin(cols, S).all(axis=1)
        expect = np.nonzero(member)[0]
        pt, found = orc.pagetable(masks, origin, shift, pool, synth.colour_set_bits(S), pool)
        assert found == expect.size and pt.tolist() == expect.tolist(), S


def test_pagetable_whole_page_closed_forms(orc):
    """M0 = bit 9 splits every 1 KiB page into colours {c, c ^ 1}; M1 = bit
    16 gives colour bit 1 = bit 6 of the page index."""
    masks = [1 << 9, 1 << 16]
    pt, found = orc.pagetable(masks, 0, 10, 256, synth.colour_set_bits([2, 3]), 256)
    assert pt.tolist() == [i for i in range(256) if (i >> 6) & 1]
    _, found = orc.pagetable(masks, 0, 10, 256, synth.colour_set_bits([0, 2]), 256)
    assert found == 0
    _, found = orc.pagetable(masks, 0, 10, 256, synth.colour_set_bits([0, 1, 2]), 256)
    assert found == 128
    # one mask inside the page: no proper subset of the colours holds a page
    for S in ([0], [1]):
        _, found = orc.pagetable([1 << 12], 0, 16, 64, synth.colour_set_bits(S), 64)
        assert found == 0
    pt, found = orc.pagetable([1 << 12], 0, 16, 64, synth.colour_set_bits([0, 1]), 64)
    assert found == 64 and pt.tolist() == list(range(64))
