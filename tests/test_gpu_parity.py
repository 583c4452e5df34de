"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bit-exact for colours, histograms, page tables, relayout and the triad;
GEMV within the fp32-accumulation bound
    |y - y_ref| <= 1e-3 * sum_k |W[m][k] x[b][k]|   and
    max|y - y_ref| / max|y_ref| <= 1e-3
against the oracle's double-precision sum.  Sizes span several tiles with
ragged tails; every seed and shape is printed before its GPU step.
"""
import sys

import numpy as np
import pytest

import synth
import paper_2407_13996_amd as sg
import gemv_cases as gc

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def ctx(orc):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = sg.Context(0)
    yield c
    c.close()


DEV = "cuda:0"

# device flags raised during each test (the gate fallback flag is not an
# error -- results stay exact -- but it should not happen; see the last test)
FLAGS = {}


@pytest.fixture(autouse=True)
def collect_flags(request, ctx):
    ctx.device_error()          # clear anything left before this test
    yield
    f = ctx.device_error()
    if f:
        FLAGS[request.node.name] = f


_SIGNED = {np.dtype(np.uint16): np.int16, np.dtype(np.uint32): np.int32,
           np.dtype(np.uint64): np.int64}


def to_dev(a: np.ndarray):
    """Upload; unsigned arrays travel as same-width signed views (raw bytes)."""
    a = np.ascontiguousarray(a)
    if a.dtype in _SIGNED:
        a = a.view(_SIGNED[a.dtype])
    return torch.from_numpy(a).to(DEV)


def to_host(t) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy()


def gemv_ok(y, ref, absdot):
    err = np.abs(y.astype(np.float64) - ref)
    assert np.all(err <= 1e-3 * absdot + 1e-30), float((err / (absdot + 1e-30)).max())
    assert err.max() <= 1e-3 * max(np.abs(ref).max(), 1e-30)


# ---------------------------------------------------------------- topology

def test_topology(ctx):
    n = ctx.num_cus
    props = torch.cuda.get_device_properties(0)
    say(f"num_cus={n} device reports {props.multi_processor_count}")
    assert n == props.multi_processor_count
    keys = [ctx.cu_key(i) for i in range(n)]
    assert len(set(keys)) == n and keys == sorted(keys)
    per_xcc = {}
    for k in keys:
        per_xcc[k >> 8] = per_xcc.get(k >> 8, 0) + 1
    say("CUs per XCC:", per_xcc)
    assert sum(per_xcc.values()) == n


# ---------------------------------------------------------------- classify

@pytest.mark.parametrize("n,K,hist", [(65536, 4, True), (65536 + 13, 6, True), (5, 8, True),
                                      (100003, 3, False), (0, 4, True), (16, 6, True),
                                      (3 * 8192 + 2048 + 31, 6, True), (8192 * 40 + 15, 1, True)])
def test_classify_matches_oracle(ctx, orc, n, K, hist):
    say(f"classify n={n} K={K} hist={hist}")
    masks = synth.xor_masks(K, seed=1, min_bit=12)
    addrs = synth.page_addresses(max(n, 1), seed=0)[:n]
    d_addrs = to_dev(addrs) if n else torch.empty(0, dtype=torch.int64, device=DEV)
    d_col = torch.full((max(n, 16) + 16,), 0xEE, dtype=torch.uint8, device=DEV)
    d_hist = torch.full((1 << K,), 12345, dtype=torch.int64, device=DEV) if hist else None
    sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist)
    got = to_host(d_col)
    ref, ref_hist = orc.classify(addrs, masks)
    assert (got[:n] == ref).all()
    assert (got[n:] == 0xEE).all()
    if hist:
        assert (to_host(d_hist).astype(np.uint64) == ref_hist).all()


def test_classify_repeated_launches_reset_histogram(ctx, orc):
    masks = synth.xor_masks(6, seed=2, min_bit=12)
    addrs = synth.page_addresses(300000, seed=3)
    d_addrs = to_dev(addrs)
    d_col = torch.empty(300016, dtype=torch.uint8, device=DEV)
    d_hist = torch.empty(64, dtype=torch.int64, device=DEV)
    _, ref_hist = orc.classify(addrs, masks)
    for i in range(3):
        sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist)
        assert (to_host(d_hist).astype(np.uint64) == ref_hist).all(), i


# ----------------------------------------------------- colour table (5.3)

def random_table(entries, seed, colours=64, holes=0.02):
    """A non-linear colour table: random colours, a few partitions with none."""
    rng = np.random.default_rng(seed)
    lut = rng.integers(0, colours, size=entries).astype(np.uint8)
    lut[rng.random(entries) < holes] = 255
    return lut


@pytest.mark.parametrize("n,shift,hist", [(65536, 10, True), (100003, 10, False),
                                          (3 * 2048 + 31, 11, True), (7, 10, True), (0, 10, True)])
def test_classify_table_matches_oracle(ctx, orc, n, shift, hist):
    say(f"classify through a colour table n={n} shift={shift} hist={hist}")
    entries, origin = 1 << 16, 1 << 34
    lut = random_table(entries, seed=n + shift)
    rng = np.random.default_rng(3)
    # most addresses inside the table, some below it and past its end
    addrs = (origin + rng.integers(-(1 << 20), (entries << shift) + (1 << 20), size=max(n, 1)))
    addrs = addrs.astype(np.uint64)[:n]
    d_lut = to_dev(lut)
    t = sg.colour_table(d_lut, origin, shift)
    d_addrs = to_dev(addrs) if n else torch.empty(0, dtype=torch.int64, device=DEV)
    d_col = torch.full((max(n, 16) + 16,), 0xEE, dtype=torch.uint8, device=DEV)
    d_hist = torch.full((256,), 777, dtype=torch.int64, device=DEV) if hist else None
    sg.colour_classify_table(ctx, t, d_addrs, d_col, d_hist)
    ref, ref_hist = orc.classify_lut(addrs, lut, origin, shift)
    got = to_host(d_col)
    assert (got[:n] == ref).all() and (got[n:] == 0xEE).all()
    if hist:
        assert (to_host(d_hist).astype(np.uint64) == ref_hist).all()


@pytest.mark.parametrize("lut_shift,page_shift,S", [(10, 10, range(32)), (10, 11, range(48)),
                                                    (10, 12, range(60)), (11, 10, [3, 7, 9, 40]),
                                                    (10, 16, range(64))])
def test_pagetable_table_matches_oracle(ctx, orc, lut_shift, page_shift, S):
    say(f"pagetable through a colour table: partitions 2^{lut_shift}, pages 2^{page_shift}")
    entries, origin = 1 << 18, 1 << 30
    lut = random_table(entries, seed=lut_shift * 31 + page_shift, holes=0.002)
    addr_origin = origin - (1 << 16)           # the pool starts before the table
    pool = ((entries << lut_shift) + (1 << 17)) >> page_shift
    words = synth.colour_set_bits(S)
    ref, ref_found = orc.pagetable_lut(lut, origin, lut_shift, addr_origin, page_shift, pool,
                                       words, pool)
    n = max(1, min(ref_found, 5000))
    d_pt = torch.full((n + 8,), -1, dtype=torch.int32, device=DEV)
    t = sg.colour_table(to_dev(lut), origin, lut_shift)
    if ref_found == 0:
        with pytest.raises(sg.SgdrcError):
            sg.colour_alloc_pagetable_table(ctx, t, addr_origin, page_shift, pool, S, n, d_pt)
        return
    found = sg.colour_alloc_pagetable_table(ctx, t, addr_origin, page_shift, pool, S, n, d_pt)
    assert found == ref_found
    got = to_host(d_pt).view(np.uint32)
    assert (got[:n] == ref[:n]).all() and (got[n:] == 0xFFFFFFFF).all()


# --------------------------------------------------------------- page table

@pytest.mark.parametrize("shift,pool,K,S,n,origin", [
    (16, 1024, 4, range(4), 64, 1 << 40),          # 4 MiB in 64 KiB pages, colours 0..3 of 16
    (12, 200003, 6, range(16), 40000, 0),
    (21, 5000, 6, range(48), 3000, 1 << 33),
    (16, 393216, 6, range(8), 3 * 16384, 1 << 36),  # three 1 GiB arrays at 8 of 64 colours
    (10, 300000, 6, range(16), 60000, 1 << 30),     # 1 KiB sectors
    (11, 100000, 6, range(24, 56), 40000, 0),       # 2 KiB sectors
])
def test_pagetable_matches_oracle(ctx, orc, shift, pool, K, S, n, origin):
    say(f"pagetable shift={shift} pool={pool} K={K} |S|={len(S)} n={n}")
    masks = synth.xor_masks(K, seed=1, min_bit=shift)
    words = synth.colour_set_bits(S)
    d_pt = torch.full((n + 8,), -1, dtype=torch.int32, device=DEV)
    found = sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, n, d_pt)
    ref, ref_found = orc.pagetable(masks, origin, shift, pool, words, n)
    assert found == ref_found
    got = to_host(d_pt).view(np.uint32)
    assert (got[:n] == ref).all()
    assert (got[n:] == 0xFFFFFFFF).all()


def test_pagetable_shortfall_reports_enomem(ctx, orc):
    masks = synth.xor_masks(4, seed=1, min_bit=16)
    d_pt = torch.zeros(1000, dtype=torch.int32, device=DEV)
    ref, ref_found = orc.pagetable(masks, 0, 16, 1000, synth.colour_set_bits([5]), 1000)
    with pytest.raises(sg.SgdrcError) as e:
        sg.colour_alloc_pagetable(ctx, masks, 0, 16, 1000, [5], 1000, d_pt)
    assert e.value.code == sg.ENOMEM and e.value.n_found == ref_found
    assert (to_host(d_pt).view(np.uint32)[:ref_found] == ref).all()


def test_pagetable_singletons_partition_the_pool(ctx):
    masks = synth.xor_masks(3, seed=9, min_bit=12)
    pool = 50000
    seen = torch.zeros(pool, dtype=torch.int32, device=DEV)
    for c in range(8):
        d_pt = torch.empty(pool, dtype=torch.int32, device=DEV)
        try:
            sg.colour_alloc_pagetable(ctx, masks, 0, 12, pool, [c], pool, d_pt)
        except sg.SgdrcError as e:
            assert e.code == sg.ENOMEM
            seen[d_pt[:e.n_found].long()] += 1
    assert bool((seen == 1).all())


@pytest.mark.parametrize("shift,lo,hi,K,S,seed", [
    (10, 8, 20, 3, [0, 1, 2, 3], 4),           # 1 KiB pages, mask bits 8..9 inside them
    (12, 10, 22, 3, [0, 1, 4, 5, 6, 7], 1),
    (16, 12, 30, 4, range(12), 6),
    (21, 16, 34, 6, range(48), 1),             # 2 MiB pages, bits 16..20 inside them
    (21, 16, 34, 6, range(48), 37),            # ... a seed where no page qualifies
    (16, 8, 40, 6, range(48), 24),             # masks on bits 8..40: no page is one colour
])
def test_pagetable_whole_pages_match_oracle(ctx, orc, shift, lo, hi, K, S, seed):
    """Masks with bits inside the page give a page's bytes several colours;
    the page qualifies only if all of them are in the set (paper section 6
    colours whole sectors).  Table and count equal the oracle's, which
    enumerates the in-page mask bits; one page more than the pool holds is
    ENOMEM with the same count."""
    masks = synth.xor_masks(K, seed=seed, min_bit=lo, hi_bit=hi)
    origin, pool = 5 << 32, 3000
    words = synth.colour_set_bits(S)
    ref, found = orc.pagetable(masks, origin, shift, pool, words, pool)
    say(f"pagetable whole pages shift={shift} mask bits {lo}..{hi} K={K}: {found} of {pool}")
    d_pt = torch.full((pool + 8,), -1, dtype=torch.int32, device=DEV)
    got_found = sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, found, d_pt)
    assert got_found == found
    got = to_host(d_pt).view(np.uint32)
    assert (got[:found] == ref).all() and (got[found:] == 0xFFFFFFFF).all()
    if found < pool:
        with pytest.raises(sg.SgdrcError) as e:
            sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, found + 1, d_pt)
        assert e.value.code == sg.ENOMEM and e.value.n_found == found


def test_pagetable_pages_hold_only_set_colours(ctx, orc):
    """Every 256-byte sub-address of every page of a GPU-built table,
    coloured by the GPU, lies in the colour set.  Mask bits 14 and 15 fall
    inside the 64 KiB pages and span colour bits 0-1, so colours 0..3 are
    whole pages: those whose address bits 17^25 and 19^30 are even, a
    quarter of the pool (closed form)."""
    masks = [(1 << 14) | (1 << 20), (1 << 15) | (1 << 22), (1 << 17) | (1 << 25),
             (1 << 19) | (1 << 30)]
    shift, pool, origin = 16, 4096, 1 << 40
    S = range(4)
    d_pt = torch.empty(pool, dtype=torch.int32, device=DEV)
    want = [i for i in range(pool) if ((i >> 1) & 1) == ((i >> 9) & 1) and ((i >> 3) & 1) == 0]
    say("pagetable colours 0..3 with in-page mask bits, then classify every 256 B")
    found = sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, len(want), d_pt)
    assert found == len(want) == pool // 4
    pt = to_host(d_pt[:found]).view(np.uint32)
    assert pt.tolist() == want
    sub = (np.uint64(origin) + (pt.astype(np.uint64)[:, None] << np.uint64(shift))
           + (np.arange(256, dtype=np.uint64) << np.uint64(8))[None, :]).reshape(-1)
    d_col = torch.empty(sub.size, dtype=torch.uint8, device=DEV)
    sg.colour_classify(ctx, masks, to_dev(sub), d_col)
    assert int(to_host(d_col).max()) <= 3
    # the same masks with the base-address rule would also take pages whose
    # other sub-addresses leave the set: colours 0..2 hold no whole page
    with pytest.raises(sg.SgdrcError) as e:
        sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, range(3), 1, d_pt)
    assert e.value.code == sg.ENOMEM and e.value.n_found == 0


@pytest.mark.parametrize("mask", [1 << 47, 1 << 10, 1 << 14, (1 << 10) | (1 << 14), 1 << 20,
                                  (1 << 21) | (1 << 23)])
def test_probe_page_sets_match_oracle(ctx, orc, mask):
    """The channel probe's page sets: the colour-0 pages of a one-mask hash
    over a 2 MiB-aligned pool of 1 KiB pages (bit 47, zero over the pool, is
    the control that keeps every page); half the pool otherwise."""
    shift, pool, origin = 10, 1 << 16, 3 << 33
    ref, found = orc.pagetable([mask], origin, shift, pool, synth.colour_set_bits([0]), pool)
    assert found == (pool if mask == 1 << 47 else pool // 2)
    say(f"probe page set, mask bits {[b for b in range(48) if (mask >> b) & 1]}")
    d_pt = torch.empty(pool, dtype=torch.int32, device=DEV)
    got = sg.colour_alloc_pagetable(ctx, [mask], origin, shift, pool, [0], found, d_pt)
    assert got == found
    assert (to_host(d_pt[:found]).view(np.uint32) == ref).all()


# ---------------------------------------------------------------- relayout

def make_tables(orc, shift, n_pages, S, seed, K=6):
    """Oracle page table of n_pages pages of colours S, and a pool size with room."""
    S = list(S)
    pool_pages = max(int(n_pages * (1 << K) / len(S) * 1.5) + 64, 1 << (K + 3))
    masks = synth.xor_masks(K, seed=seed, min_bit=shift)
    pt, found = orc.pagetable(masks, 0, shift, pool_pages, synth.colour_set_bits(S), n_pages)
    assert found >= n_pages
    return pt, pool_pages


@pytest.mark.parametrize("shift,n_bytes", [(12, 37 * 4096 + 1234), (16, 9 * 65536 + 17),
                                           (21, 2 * 2097152 + 4096 * 3 + 5), (15, 1),
                                           (16, 64 * 65536), (14, 11 * 16384 + 4015),
                                           (13, 15), (17, 3 * 131072 + 65536 + 32),
                                           (10, 37 * 1024 + 77), (11, 19 * 2048 + 1500)])
def test_relayout_matches_oracle(ctx, orc, shift, n_bytes):
    say(f"relayout shift={shift} n_bytes={n_bytes}")
    P = 1 << shift
    n_pages = -(-n_bytes // P)
    pt_s, src_pages = make_tables(orc, shift, n_pages, range(16), 1)
    pt_d, dst_pages = make_tables(orc, shift, n_pages, range(16, 48), 2)
    src = synth.random_bytes(src_pages * P, seed=3)
    dst0 = synth.random_bytes(dst_pages * P, seed=4)
    d_src, d_dst = to_dev(src), to_dev(dst0)
    sg.bimodal_relayout(ctx, sg.paged(d_dst, to_dev(pt_d), dst_pages),
                        sg.paged(d_src, to_dev(pt_s), src_pages), n_bytes, shift)
    ref = dst0.copy()
    orc.relayout(ref, pt_d, src, pt_s, n_bytes, shift)
    assert (to_host(d_dst) == ref).all()


@pytest.mark.parametrize("n_items,cus", [(40, None), (7, 37)])
def test_relayout_batch_matches_oracle(ctx, orc, n_items, cus):
    """Batched relayout: items of mixed page sizes and ragged lengths (one
    empty, some shorter than 16 bytes, some spanning several tiles), more
    than one launch's worth of items, and under a random CU subset; each item
    equals the oracle's relayout, dst bytes past n_bytes untouched."""
    rng = np.random.default_rng(n_items)
    shifts = [10, 12, 16, 10, 12, 16, 21, 16]
    items, refs, devs, keep = [], [], [], []
    for i in range(n_items):
        shift = shifts[i % len(shifts)]
        P = 1 << shift
        kind = i % 5
        n_bytes = (0 if i == 3 else int(rng.integers(1, 16)) if kind == 1
                   else int(rng.integers(1, 3 * 65536 + 100)) if kind != 4
                   else int(rng.integers(3 * 65536, 9 * 65536)))
        n_pages = max(1, -(-n_bytes // P))
        pt_s, src_pages = make_tables(orc, shift, n_pages, range(16), 10 + i)
        pt_d, dst_pages = make_tables(orc, shift, n_pages, range(32, 48), 60 + i)
        src = synth.random_bytes(src_pages * P, seed=100 + i)
        dst0 = synth.random_bytes(dst_pages * P, seed=200 + i)
        d_src, d_dst, d_ps, d_pd = to_dev(src), to_dev(dst0), to_dev(pt_s), to_dev(pt_d)
        keep += [d_src, d_ps, d_pd]
        items.append((sg.paged(d_dst, d_pd, dst_pages), sg.paged(d_src, d_ps, src_pages),
                      n_bytes, shift))
        ref = dst0.copy()
        orc.relayout(ref, pt_d, src, pt_s, n_bytes, shift)
        refs.append(ref)
        devs.append(d_dst)
    say(f"relayout batch of {n_items} items on {'all' if cus is None else cus} CUs")
    if cus is not None:
        sg.set_cu_mask(ctx, None, synth.random_cu_subset(ctx.num_cus, cus, seed=9))
    try:
        sg.bimodal_relayout_batch(ctx, items)
    finally:
        sg.set_cu_mask(ctx, None, None)
    for i, (d, ref) in enumerate(zip(devs, refs)):
        assert (to_host(d) == ref).all(), i


def test_relayout_round_trip_fp16_is_identity(ctx, orc):
    shift = 16
    n_pages = 300
    n_bytes = n_pages * 65536 - 6
    data = synth.random_u16(n_pages * 32768, seed=5)
    d_all = to_dev(data)
    pt_all = torch.arange(n_pages, dtype=torch.int32, device=DEV)
    pt_s, pool_s = make_tables(orc, shift, n_pages, range(16), 3)
    pt_s = to_dev(pt_s)
    d_s = torch.zeros(pool_s * 32768, dtype=torch.int16, device=DEV)
    d_back = torch.zeros_like(d_all)
    sg.bimodal_relayout(ctx, sg.paged(d_s, pt_s, pool_s), sg.paged(d_all, pt_all, n_pages),
                        n_bytes, shift)
    sg.bimodal_relayout(ctx, sg.paged(d_back, pt_all, n_pages), sg.paged(d_s, pt_s, pool_s),
                        n_bytes, shift)
    back = to_host(d_back).view(np.uint16)
    assert (back[:n_bytes // 2] == data[:n_bytes // 2]).all()
    assert (back[n_bytes // 2:] == 0).all()


# ------------------------------------------------------------------- triad

@pytest.mark.parametrize("shift,n", [(12, 5 * 1024 + 77), (16, 3 * 16384 + 5), (16, 40 * 16384),
                                     (21, 524288 + 3), (13, 7), (14, 9 * 4096 + 2),
                                     (15, 5 * 8192 + 1), (16, 3), (10, 9 * 256 + 3),
                                     (11, 40 * 512 + 1), (10, 600 * 256)])
def test_triad_matches_oracle(ctx, orc, shift, n):
    say(f"triad shift={shift} n={n}")
    P = 1 << shift
    n_pages = -(-n * 4 // P)
    tabs = [make_tables(orc, shift, n_pages, range(8 * i, 8 * i + 16), 10 + i) for i in range(3)]
    pools = max(t[1] for t in tabs)
    pts = [t[0] for t in tabs]
    epp = P // 4
    a0 = synth.uniform_f32(pools * epp, seed=1)
    b = synth.uniform_f32(pools * epp, seed=2)
    c = synth.uniform_f32(pools * epp, seed=3)
    d_a, d_b, d_c = to_dev(a0), to_dev(b), to_dev(c)
    sg.colored_stream(ctx, sg.paged(d_a, to_dev(pts[0]), pools), sg.paged(d_b, to_dev(pts[1]), pools),
                      sg.paged(d_c, to_dev(pts[2]), pools), 3.0, n, shift)
    ref = a0.copy()
    orc.triad(ref, pts[0], b, pts[1], c, pts[2], 3.0, n, shift)
    assert (to_host(d_a).view(np.uint32) == ref.view(np.uint32)).all()


def test_triad_in_place_alias(ctx, orc):
    shift, n = 16, 10 * 16384 + 3
    pages = 11
    pt = torch.arange(pages, dtype=torch.int32, device=DEV)
    b = synth.uniform_f32(pages * 16384, seed=7)
    c = synth.uniform_f32(pages * 16384, seed=8)
    d_b, d_c = to_dev(b), to_dev(c)
    sg.colored_stream(ctx, sg.paged(d_b, pt, pages), sg.paged(d_b, pt, pages),
                      sg.paged(d_c, pt, pages), -0.5, n, shift)
    ref = b.copy()
    ident = np.arange(pages, dtype=np.uint32)
    orc.triad(ref, ident, b, ident, c, ident, -0.5, n, shift)
    assert (to_host(d_b).view(np.uint32) == ref.view(np.uint32)).all()


# ----------------------------------------------- full-size configurations

def aligned_pool(n_pages, shift):
    """A device byte pool of n_pages pages whose base is page aligned."""
    P = 1 << shift
    raw = torch.empty(n_pages * P + P, dtype=torch.uint8, device=DEV)
    off = (-raw.data_ptr()) % P
    return raw, raw.data_ptr() + off, off


def test_classify_2e26_addresses_full_size(ctx, orc):
    """2^26 random 4 KiB-aligned addresses, 6 masks: every colour and the
    histogram equal the oracle's."""
    n = 1 << 26
    masks = synth.xor_masks(6, seed=1, min_bit=12)
    addrs = synth.page_addresses(n, seed=0)
    d_col = torch.full((n + 16,), 0xEE, dtype=torch.uint8, device=DEV)
    d_hist = torch.zeros(64, dtype=torch.int64, device=DEV)
    say("classify 2^26 addresses")
    sg.colour_classify(ctx, masks, to_dev(addrs), d_col, d_hist)
    ref, ref_hist = orc.classify(addrs, masks)
    got = to_host(d_col)
    assert (got[:n] == ref).all() and (got[n:] == 0xEE).all()
    assert (to_host(d_hist).astype(np.uint64) == ref_hist).all()


@pytest.mark.parametrize("elems,colours,cus", [
    (1 << 28, range(8), None),               # three 1 GiB arrays at 8 of 64 colours, all CUs
    (1 << 29, range(48, 64), range(192, 256)),  # the co-located pair's BE stream: 2 GiB arrays, 64 CUs
])
def test_triad_full_size_sampled(ctx, orc, elems, colours, cus):
    """Full-size triad through GPU-built page tables (compared with the
    oracle's in full); 2^18 sampled elements of a against the oracle's fmaf."""
    shift, P = 16, 1 << 16
    epp = P // 4
    pages = elems // epp
    masks = synth.xor_masks(6, seed=1, min_bit=shift)
    colours = list(colours)
    pool_pages = int(3 * pages * 64 / len(colours) * 1.04) + 64
    raw, base, off = aligned_pool(pool_pages, shift)
    say(f"triad {elems} elements, {len(colours)}/64 colours, pool {pool_pages} pages")
    d_pt = torch.empty(3 * pages, dtype=torch.int32, device=DEV)
    sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_pages, colours, 3 * pages, d_pt)
    ref_pt, found = orc.pagetable(masks, base, shift, pool_pages, synth.colour_set_bits(colours),
                                  3 * pages)
    assert found >= 3 * pages
    assert (to_host(d_pt).view(np.uint32) == ref_pt).all()
    pts = [d_pt[i * pages:(i + 1) * pages] for i in range(3)]
    arr = [sg.paged(base, pts[i], pool_pages) for i in range(3)]
    b = synth.uniform_f32(elems, seed=2)
    c = synth.uniform_f32(elems, seed=3)
    ident = torch.arange(pages, dtype=torch.int32, device=DEV)
    d_b, d_c = to_dev(b), to_dev(c)
    sg.bimodal_relayout(ctx, arr[1], sg.paged(d_b, ident, pages), elems * 4, shift)
    sg.bimodal_relayout(ctx, arr[2], sg.paged(d_c, ident, pages), elems * 4, shift)
    del d_b, d_c
    stream = torch.cuda.current_stream()
    if cus is not None:
        sg.set_cu_mask(ctx, stream, cus)
    try:
        sg.colored_stream(ctx, arr[0], arr[1], arr[2], 3.0, elems, shift, stream)
    finally:
        sg.set_cu_mask(ctx, stream, None)
    rng = np.random.default_rng(11)
    idx = np.sort(rng.choice(elems, size=1 << 18, replace=False)).astype(np.int64)
    pa = ref_pt[:pages].astype(np.int64)
    where = off // 4 + pa[idx // epp] * epp + idx % epp       # float index into raw
    got = to_host(raw.view(torch.float32)[torch.from_numpy(where).to(DEV)])
    k = idx.size
    kp = -(-k // epp)
    bs = np.zeros(kp * epp, np.float32); bs[:k] = b[idx]
    cs = np.zeros(kp * epp, np.float32); cs[:k] = c[idx]
    ref = np.zeros(kp * epp, np.float32)
    ident_h = np.arange(kp, dtype=np.uint32)
    orc.triad(ref, ident_h, bs, ident_h, cs, ident_h, 3.0, k, shift)
    assert (got.view(np.uint32) == ref[:k].view(np.uint32)).all()


def test_relayout_4gib_fp16_full_size(ctx, orc):
    """4 GiB fp16 tensor (65,536 pages of 64 KiB) from the all-colour page set
    to 16 of 64 colours and back: every restricted page holds its source page
    at the oracle table's position, and the round trip is the identity."""
    shift, P = 16, 1 << 16
    pages = 65536
    n_bytes = pages * P
    masks = synth.xor_masks(6, seed=1, min_bit=shift)
    colours = list(range(16))
    pool_pages = int(pages * 4 * 1.04) + 64
    raw, base, off = aligned_pool(pool_pages, shift)
    ref_pt, found = orc.pagetable(masks, base, shift, pool_pages, synth.colour_set_bits(colours),
                                  pages)
    assert found >= pages
    d_pt = to_dev(ref_pt)
    g = torch.Generator(device=DEV)
    g.manual_seed(5)
    src = torch.randint(-32768, 32768, (n_bytes // 2,), generator=g, dtype=torch.int16, device=DEV)
    ident = torch.arange(pages, dtype=torch.int32, device=DEV)
    say("relayout 4 GiB all -> 16/64 -> all")
    sg.bimodal_relayout(ctx, sg.paged(base, d_pt, pool_pages), sg.paged(src, ident, pages),
                        n_bytes, shift)
    pool_pages_view = raw[off:off + pool_pages * P].view(pool_pages, P)
    rows = torch.from_numpy(ref_pt.astype(np.int64)).to(DEV)
    same = 0
    for j0 in range(0, pages, 8192):      # compare in 512 MiB slices
        sel = rows[j0:j0 + 8192]
        same += int((pool_pages_view.index_select(0, sel)
                     == src.view(torch.uint8).view(pages, P)[j0:j0 + 8192]).all().item())
    assert same == pages // 8192
    back = torch.zeros_like(src)
    sg.bimodal_relayout(ctx, sg.paged(back, ident, pages), sg.paged(base, d_pt, pool_pages),
                        n_bytes, shift)
    torch.cuda.synchronize()
    assert bool(torch.equal(back, src))


# -------------------------------------------------------------------- GEMV

def w_bits(dt, n, seed):
    if dt == sg.F32:
        return synth.normal_f32(n, seed=seed).view(np.uint32)
    if dt == sg.BF16:
        return synth.normal_bf16(n, seed=seed, sigma=0.02)
    return synth.normal_f32(n, seed=seed, sigma=0.5).astype(np.float16).view(np.uint16)


def x_bits(dt, n, seed):
    if dt == sg.F32:
        return synth.normal_f32(n, seed=seed).view(np.uint32)
    if dt == sg.BF16:
        return synth.normal_bf16(n, seed=seed)
    return synth.normal_f32(n, seed=seed).astype(np.float16).view(np.uint16)


def cu_list(cus):
    """None (all CUs), a count n (the first n logical CUs) or a list."""
    if cus is None or isinstance(cus, (list, range)):
        return cus
    return range(cus)


ERR_LOG = {}


def gemv_check(ctx, y, ref, absdot, M, K, B, wd, xd, cus, tag=""):
    """The 1e-3 criterion, and the tighter bound of the kernel's own
    summation tree: |y - ref| <= 2 * depth * 2^-24 * sum|W x| with depth the
    plan's sum_depth (each of at most depth fp32 roundings errs by at most
    one unit, or two if a step rounds towards zero)."""
    gemv_ok(y, ref, absdot)
    n = ctx.num_cus if cus is None else len(list(cus))
    depth = sg.gemv_plan(n, wd, M, K, xd, B)["sum_depth"]
    err = np.abs(y.astype(np.float64) - ref)
    ratio = err / (absdot + 1e-30)
    ERR_LOG[(M, K, B, wd, xd, n, tag)] = (float(ratio.max()), depth)
    say(f"  max |err| / sum|Wx| = {ratio.max():.3g} (bound {2 * depth * 2.0 ** -24:.3g}, "
        f"depth {depth})")
    assert np.all(err <= 2 * depth * 2.0 ** -24 * absdot + 1e-30), float(ratio.max())


def upload_w(orc, M, K, wd, shift, S, seed, masks_seed, n_masks):
    """W [M x K] of dtype wd placed on an oracle page table of colours S;
    returns host pool and table, device pool and table, and the pool size."""
    P = 1 << shift
    wb = w_bits(wd, M * K, seed + 1)
    wbytes = wb.view(np.uint8)
    n_pages = -(-wbytes.size // P)
    pt, pool_pages = make_tables(orc, shift, n_pages, S, masks_seed, K=n_masks)
    pool = np.zeros(pool_pages * P, dtype=np.uint8)
    padded = np.zeros(n_pages * P, dtype=np.uint8)
    padded[:wbytes.size] = wbytes
    pool.reshape(pool_pages, P)[pt.astype(np.int64)] = padded.reshape(n_pages, P)
    return pool, pt, to_dev(pool), to_dev(pt), pool_pages


def launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, wd, xd, d_x, shift, cus):
    d_y = torch.full((B * M,), float("nan"), dtype=torch.float32, device=DEV)
    if cus is not None:
        sg.set_cu_mask(ctx, None, cus)
    try:
        sg.colored_gemv(ctx, sg.paged(d_pool, d_pt, pool_pages), wd, M, K, d_x, xd, B, d_y, shift)
    finally:
        if cus is not None:
            sg.set_cu_mask(ctx, None, None)
    return to_host(d_y).reshape(B, M)


def run_gemv(ctx, orc, M, K, B, wd, xd, shift, S=range(48), seed=0, masks_seed=1, cus=None,
             check=True, n_masks=6):
    cus = cu_list(cus)
    pool, pt, d_pool, d_pt, pool_pages = upload_w(orc, M, K, wd, shift, S, seed, masks_seed,
                                                  n_masks)
    xb = x_bits(xd, B * K, seed + 2)
    y = launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, wd, xd, to_dev(xb), shift, cus)
    if check:
        ref, absdot = orc.gemv(pool, pt, wd, M, K, xb, xd, B, shift)
        gemv_check(ctx, y, ref, absdot, M, K, B, wd, xd, cus)
    return y


def _case_id(c):
    M, K, B, wd, xd, shift, cus = c
    return f"{M}x{K}-B{B}-w{wd}x{xd}-p{1 << (shift - 10)}K-cus{cus}"


def test_gemv_fp32_1024x1024(ctx, orc):
    say("gemv 1024x1024 fp32 B=1, 64 KiB pages, colours 0..3 of 16")
    run_gemv(ctx, orc, 1024, 1024, 1, sg.F32, sg.F32, 16, S=range(4), n_masks=4)


@pytest.mark.parametrize("case", gc.RAGGED + gc.DTYPE_MIX + gc.STAGING + gc.MFMA_CHUNKS
                         + gc.LONG_ROWS + gc.SECTORS + gc.SINGLE_ROWS + gc.PAGE_EDGES + gc.X_STAGED,
                         ids=_case_id)
def test_gemv_matches_oracle(ctx, orc, case):
    """Ragged shapes (1003 x 1000, batches 1..8), mixed dtypes, W tables of
    256 pages (staged once per workgroup) and 257 (staged per tile), MFMA
    chunk counts (odd, ragged last chunk, rows far shorter than a chunk),
    long rows at batch 1 on few and many CUs, 1-2 KiB sector pages,
    single-row matrices (most of the tile outside M), and 2 MiB pages with
    tiles inside one page (per-row buffer resources on the MFMA path) beside
    tiles that straddle a page end (a table read per load)."""
    M, K, B, wd, xd, shift, cus = case
    say(f"gemv {_case_id(case)}")
    run_gemv(ctx, orc, M, K, B, wd, xd, shift, seed=M + K + B + shift, cus=cus)


@pytest.mark.parametrize("M,K,B,cus,dt", gc.HALF_TILES)
def test_gemv_mfma_half_tiles(ctx, orc, M, K, B, cus, dt):
    """The MFMA path takes 8-row tiles (upper half of the A operand zero)
    when they leave the busiest CU fewer rows than 16-row tiles: a ragged
    last tile, the 4096 x 11008 layer on 192 CUs, two CUs.  A mask of one CU
    per 16-row tile (16-row tiles there) gives the same bits."""
    say(f"gemv mfma {M}x{K} B={B} dtype {dt} on {cus} CUs (8-row tiles)")
    y8 = run_gemv(ctx, orc, M, K, B, dt, dt, 16, seed=M + B, cus=cus)
    t16 = -(-M // 16)
    assert t16 <= ctx.num_cus
    y16 = run_gemv(ctx, orc, M, K, B, dt, dt, 16, seed=M + B, cus=range(t16), check=False)
    assert (y8.view(np.uint32) == y16.view(np.uint32)).all()


@pytest.mark.parametrize("case", gc.X_ONCE, ids=_case_id)
def test_gemv_x_once_matches_oracle_and_per_tile_x(ctx, orc, case):
    """Vector path with x loaded once per workgroup (rows that one round of
    loads covers, x half a tile's bytes; f16 and bf16, a K tail inside the
    round, 4 KiB pages) against the oracle.  The same x values passed as
    fp32 take the same tile shape with x loaded per tile (W and x differ in
    type), and their products are exact, so the bits must match."""
    M, K, B, wd, xd, shift, cus = case
    p = sg.gemv_plan(cus or ctx.num_cus, wd, M, K, xd, B)
    assert p["x_once"], p
    say(f"gemv x once {_case_id(case)}")
    seed = M + K + B
    pool, pt, d_pool, d_pt, pool_pages = upload_w(orc, M, K, wd, shift, range(48), seed, 1, 6)
    xb = x_bits(xd, B * K, seed + 2)
    y = launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, wd, xd, to_dev(xb), shift, cu_list(cus))
    ref, absdot = orc.gemv(pool, pt, wd, M, K, xb, xd, B, shift)
    gemv_check(ctx, y, ref, absdot, M, K, B, wd, xd, cu_list(cus))
    if xd == sg.BF16:
        xf = (xb.astype(np.uint32) << 16).view(np.float32)
    else:
        xf = xb.view(np.float16).astype(np.float32)
    q = sg.gemv_plan(cus or ctx.num_cus, wd, M, K, sg.F32, B)
    assert not q["x_once"] and (q["rows"], q["loads"]) == (p["rows"], p["loads"]), (p, q)
    y2 = launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, wd, sg.F32, to_dev(xf.view(np.uint32)),
                     shift, cu_list(cus))
    assert (y.view(np.uint32) == y2.view(np.uint32)).all()


@pytest.mark.parametrize("dt", [sg.BF16, sg.F16], ids=["bf16", "f16"])
def test_gemv_mfma_x_rows_same_bits(ctx, orc, dt):
    """The MFMA path stages four rows of x at batch 3-4 and eight at batch
    5-8 (here at batch 3-4 for the whole K at once, skipping the pad chunk,
    at batch 5-8 chunk by chunk).  A batch column's sums do not depend on
    the other columns, so the first rows of batch-5 and batch-8 launches
    equal batch-3 and batch-4 launches over the same rows of x bit for bit;
    each launch also matches the oracle (1003 x 1000: a ragged last tile
    and a ragged last chunk)."""
    M, K, shift = 1003, 1000, 16
    say(f"gemv mfma {M}x{K} dtype {dt}: batches 3, 4, 5, 8 over shared rows of x")
    pool, pt, d_pool, d_pt, pool_pages = upload_w(orc, M, K, dt, shift, range(48), 7, 1, 6)
    xb = x_bits(dt, 8 * K, 9)
    ys = {}
    for B in (3, 4, 5, 8):
        p = sg.gemv_plan(ctx.num_cus, dt, M, K, dt, B)
        assert p["path"] == "mfma" and p["batch_cols"] == (4 if B <= 4 else 8), p
        assert p["x_once"] == (B <= 4), p   # whole-K x in LDS at batch 3-4 (rows of 2000 bytes)
        x = np.ascontiguousarray(xb[:B * K])
        ys[B] = launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, dt, dt, to_dev(x), shift, None)
        ref, absdot = orc.gemv(pool, pt, dt, M, K, x, dt, B, shift)
        gemv_check(ctx, ys[B], ref, absdot, M, K, B, dt, dt, None, tag=f"batch {B}")
    for lo, hi in ((3, 5), (4, 8), (3, 8)):
        assert (ys[lo].view(np.uint32) == ys[hi][:lo].view(np.uint32)).all(), (lo, hi)


def test_zero_length_triad_and_relayout_touch_nothing(ctx):
    shift, P = 16, 65536
    pt = torch.zeros(1, dtype=torch.int32, device=DEV)
    a = torch.full((P // 4,), 7.0, dtype=torch.float32, device=DEV)
    b = torch.ones(P // 4, dtype=torch.float32, device=DEV)
    sg.colored_stream(ctx, sg.paged(a, pt, 1), sg.paged(b, pt, 1), sg.paged(b, pt, 1), 3.0, 0, shift)
    dst = torch.full((P,), 5, dtype=torch.uint8, device=DEV)
    src = torch.zeros(P, dtype=torch.uint8, device=DEV)
    sg.bimodal_relayout(ctx, sg.paged(dst, pt, 1), sg.paged(src, pt, 1), 0, shift)
    sg.bimodal_relayout_batch(ctx, [])
    assert (to_host(a) == 7.0).all()
    assert (to_host(dst) == 5).all()


LS_CACHE = {}


@pytest.fixture(scope="module")
def ls_weights(orc):
    """The two LS layers, 4096x11008 and 11008x4096 (bf16, N(0, 0.02)) in 2 MiB pages on colours 0..47
    of 64, uploaded once; freed at the end of the module."""
    def get(M, K):
        if (M, K) not in LS_CACHE:
            LS_CACHE.clear()
            torch.cuda.empty_cache()
            LS_CACHE[(M, K)] = upload_w(orc, M, K, sg.BF16, 21, range(48), seed=M, masks_seed=1,
                                        n_masks=6)
        return LS_CACHE[(M, K)]
    yield get
    LS_CACHE.clear()


@pytest.mark.parametrize("M,K", gc.LS_LAYERS)
@pytest.mark.parametrize("B", gc.LS_BATCHES)
def test_gemv_ls_layers_sweep(ctx, orc, ls_weights, M, K, B):
    """The full sweep of the LS layers: both at their real size (bf16, 2 MiB pages
    on colours 0..47) at every batch on the first 64/128/192/256 CUs -- every
    kernel variant the benchmark times for this configuration (vector path
    with 2-, 4- and 8-row tiles, MFMA with 8- and 16-row tiles).  Each
    result is within the oracle bound and bitwise equal across the masks."""
    pool, pt, d_pool, d_pt, pool_pages = ls_weights(M, K)
    xb = x_bits(sg.BF16, B * K, M + B + 2)
    d_x = to_dev(xb)
    ref, absdot = orc.gemv(pool, pt, sg.BF16, M, K, xb, sg.BF16, B, 21)
    ys = []
    for n in gc.LS_CUS:
        if n > ctx.num_cus:
            continue
        plan = sg.gemv_plan(n, sg.BF16, M, K, sg.BF16, B)
        say(f"gemv LS layer {M}x{K} B={B} on {n} CUs: {plan['path']} rows {plan['rows']} "
            f"loads {plan['loads']}")
        y = launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, sg.BF16, sg.BF16, d_x, 21,
                        range(n))
        gemv_check(ctx, y, ref, absdot, M, K, B, sg.BF16, sg.BF16, range(n), tag="c3")
        ys.append(y)
    for y in ys[1:]:
        assert (y.view(np.uint32) == ys[0].view(np.uint32)).all()


def test_gemv_bitwise_identical_across_cu_masks(ctx, orc):
    n = ctx.num_cus
    ys = []
    for cus in [None, range(64), range(n // 2, n), synth.random_cu_subset(n, 37, seed=4)]:
        say(f"gemv mask {None if cus is None else len(list(cus))} CUs")
        for B in (1, 8):
            ys.append((B, run_gemv(ctx, orc, 777, 2048, B, sg.BF16, sg.BF16, 16, seed=B,
                                   cus=cus, check=(cus is None))))
    for B in (1, 8):
        same = [y for b, y in ys if b == B]
        for y in same[1:]:
            assert (y.view(np.uint32) == same[0].view(np.uint32)).all()


@pytest.mark.parametrize("M,K,B", [(4096, 11008, 1), (11008, 4096, 8), (777, 2048, 2), (5, 64, 1)])
def test_gemv_static_schedule_visits_each_tile_once(ctx, orc, M, K, B):
    """Masks of whole XCDs (all CUs, the first 32/96/192 CUs, XCDs 1 and 6)
    take the static schedule, any other mask the ticket queues: every tile is
    taken exactly once, only by allowed CUs, and the output bits are the same
    under every mask."""
    n = ctx.num_cus
    x_count = n // 32
    shift = 21 if M * K * 2 >= (1 << 24) else 12
    pool, pt, d_pool, d_pt, pool_pages = upload_w(orc, M, K, sg.BF16, shift, range(48), M + K,
                                                  1, 6)
    xb = x_bits(sg.BF16, B * K, M + 3)
    d_x = to_dev(xb)
    ref, absdot = orc.gemv(pool, pt, sg.BF16, M, K, xb, sg.BF16, B, shift)
    stream = torch.cuda.current_stream()
    masks = [(None, "static"), (range(32), "static"), (range(96), "static"),
             (list(range(32, 64)) + list(range(192, 224)), "static"),
             (range(100), "queue"), (synth.random_cu_subset(n, 37, seed=8), "queue")]
    ys = []
    for cus, want in masks:
        cl_ = torch.zeros(n, dtype=torch.int32, device=DEV)
        tiles_cap = M + 64
        tl_ = torch.zeros(tiles_cap, dtype=torch.int32, device=DEV)
        ctx.set_worklog(cl_, tl_)
        try:
            y = launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, sg.BF16, sg.BF16, d_x, shift, cus)
            tiles = ctx.last_tiles(stream)
            sched = ctx.last_schedule(stream)
        finally:
            ctx.set_worklog(None, None)
        say(f"gemv {M}x{K} B={B} mask {'all' if cus is None else len(list(cus))}: {sched}, "
            f"{tiles} tiles")
        assert x_count != 8 or sched == want
        cl, tl = to_host(cl_), to_host(tl_)
        assert (tl[:tiles] == 1).all() and (tl[tiles:] == 0).all()
        allowed = set(range(n)) if cus is None else set(cus)
        assert set(np.nonzero(cl)[0].tolist()) <= allowed and cl.sum() == tiles
        gemv_check(ctx, y, ref, absdot, M, K, B, sg.BF16, sg.BF16, cus, tag="sched")
        ys.append(y)
    for y in ys[1:]:
        assert (y.view(np.uint32) == ys[0].view(np.uint32)).all()


def test_gemv_timelog_static_schedule(ctx, orc):
    """The time log of statically scheduled GEMVs: the end stamp is the
    largest of the workgroups' partial stamps (reduced after each launch and
    cleared), so every span is positive and within the host-event time."""
    M, K = 4096, 11008
    pool, pt, d_pool, d_pt, pool_pages = upload_w(orc, M, K, sg.BF16, 21, range(48), 1, 1, 6)
    d_x = to_dev(x_bits(sg.BF16, K, 2))
    d_y = torch.empty(M, dtype=torch.float32, device=DEV)
    stream = torch.cuda.current_stream()
    slots = torch.zeros(2 * 4, dtype=torch.int64, device=DEV)
    khz = ctx.wallclock_khz
    ctx.set_timelog(stream, slots)
    spans = []
    try:
        for i in range(8):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            sg.colored_gemv(ctx, sg.paged(d_pool, d_pt, pool_pages), sg.BF16, M, K, d_x, sg.BF16,
                            1, d_y, 21, stream)
            e1.record(stream)
            torch.cuda.synchronize()
            assert ctx.last_schedule(stream) == "static"
            t = to_host(slots).astype(np.int64).reshape(4, 2)[i % 4]
            span = (int(t[1]) - int(t[0])) / khz
            spans.append(span)
            assert 0 < span <= e0.elapsed_time(e1) + 0.01, (span, e0.elapsed_time(e1))
    finally:
        ctx.set_timelog(stream, None)
    say(f"  static GEMV spans (us): {[round(x * 1e3, 1) for x in spans]}")


# ------------------------------------------------------------- time log

def test_timelog_brackets_each_launch(ctx):
    """Each gated launch stamps {start, end} device-clock ticks into its slot
    (slots used cyclically); the span is positive and no longer than the
    host-event time around the same launch."""
    import torch
    shift, elems = 16, 64 * 16384
    pages = elems * 4 >> shift
    pt = torch.arange(pages, dtype=torch.int32, device=DEV)
    b = to_dev(synth.uniform_f32(elems, seed=1))
    c = to_dev(synth.uniform_f32(elems, seed=2))
    a = torch.zeros_like(b)
    stream = torch.cuda.current_stream()
    slots = torch.zeros(2 * 3, dtype=torch.int64, device=DEV)
    khz = ctx.wallclock_khz
    assert khz > 0
    ctx.set_timelog(stream, slots)
    spans = []
    for i in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        sg.colored_stream(ctx, sg.paged(a, pt, pages), sg.paged(b, pt, pages),
                          sg.paged(c, pt, pages), 2.0, elems, shift, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        t = to_host(slots).astype(np.int64).reshape(3, 2)[i % 3]
        span_ms = (int(t[1]) - int(t[0])) / khz
        spans.append(span_ms)
        assert 0 < span_ms <= e0.elapsed_time(e1) + 0.05, (span_ms, e0.elapsed_time(e1))
    ctx.set_timelog(stream, None)
    before = to_host(slots).copy()
    sg.colored_stream(ctx, sg.paged(a, pt, pages), sg.paged(b, pt, pages),
                      sg.paged(c, pt, pages), 2.0, elems, shift, stream)
    torch.cuda.synchronize()
    assert (to_host(slots) == before).all()
    say(f"  time-log spans (ms): {[round(x, 4) for x in spans]}")


# ------------------------------------------------------- CU gate and queue

def test_cu_mask_confines_work_and_visits_each_tile_once(ctx, orc):
    n = ctx.num_cus
    shift, elems = 16, 600 * 16384
    pages = elems * 4 >> shift
    pt = torch.arange(pages, dtype=torch.int32, device=DEV)
    b = to_dev(synth.uniform_f32(elems, seed=1))
    c = to_dev(synth.uniform_f32(elems, seed=2))
    ref = None
    stream = torch.cuda.current_stream()
    for cus in [list(range(64)), list(range(128, n)), synth.random_cu_subset(n, 20, seed=3),
                list(range(n)), [5]]:
        say(f"gate mask of {len(cus)} CUs")
        a = torch.zeros_like(b)
        cu_log = torch.zeros(n, dtype=torch.int32, device=DEV)
        tile_log = torch.zeros(4096, dtype=torch.int32, device=DEV)
        ctx.set_worklog(cu_log, tile_log)
        sg.set_cu_mask(ctx, stream, cus)
        sg.colored_stream(ctx, sg.paged(a, pt, pages), sg.paged(b, pt, pages),
                          sg.paged(c, pt, pages), 3.0, elems, shift, stream)
        tiles = ctx.last_tiles(stream)
        ctx.set_worklog(None, None)
        sg.set_cu_mask(ctx, stream, None)
        assert ctx.device_error() & sg.DEVERR_PT_RANGE == 0
        cl, tl = to_host(cu_log), to_host(tile_log)
        assert tiles == elems * 4 // 65536  # 64 KiB stream tiles
        assert (tl[:tiles] == 1).all() and (tl[tiles:] == 0).all()
        worked = set(np.nonzero(cl)[0].tolist())
        assert worked <= set(cus)
        assert cl.sum() == tiles
        say(f"  {len(worked)} of {len(cus)} allowed CUs took tiles")
        out = to_host(a)
        if ref is None:
            ref = out
        assert (out.view(np.uint32) == ref.view(np.uint32)).all()


def test_classify_wavefront_tiles_under_cu_masks(ctx, orc):
    """Classify hands its tiles (1024 addresses) to single wavefronts, by the
    static schedule under masks of whole XCDs (adjacent or not) and through
    the ticket queues otherwise: under every mask each tile is taken once,
    only allowed CUs work, and colours and histogram equal the oracle's."""
    n_cu = ctx.num_cus
    n = (1 << 20) + 37
    masks = synth.xor_masks(6, seed=5, min_bit=12)
    addrs = synth.page_addresses(n, seed=6)
    ref, ref_hist = orc.classify(addrs, masks)
    d_addrs = to_dev(addrs)
    stream = torch.cuda.current_stream()
    tiles_expected = (n & ~15) // 1024 + (1 if (n & ~15) % 1024 else 0)
    whole_xcds = n_cu == 256   # masks of whole XCDs take the static schedule
    for cus, want in [(list(range(64)), "static"), (synth.random_cu_subset(n_cu, 20, seed=8), "queue"),
                      ([5], "queue"), ([n_cu - 1], "queue"), (list(range(n_cu)), "static"),
                      (list(range(32, 64)) + list(range(192, 224)), "static")]:
        say(f"classify under a mask of {len(cus)} CUs")
        d_col = torch.full((n + 16,), 0xEE, dtype=torch.uint8, device=DEV)
        d_hist = torch.zeros(64, dtype=torch.int64, device=DEV)
        cu_log = torch.zeros(n_cu, dtype=torch.int32, device=DEV)
        tile_log = torch.zeros(4096, dtype=torch.int32, device=DEV)
        ctx.set_worklog(cu_log, tile_log)
        sg.set_cu_mask(ctx, stream, cus)
        sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist, stream)
        tiles = ctx.last_tiles(stream)
        sched = ctx.last_schedule(stream)
        ctx.set_worklog(None, None)
        sg.set_cu_mask(ctx, stream, None)
        cl, tl = to_host(cu_log), to_host(tile_log)
        assert tiles == tiles_expected
        assert not whole_xcds or sched == want, (len(cus), sched)
        assert (tl[:tiles] == 1).all() and (tl[tiles:] == 0).all()
        assert set(np.nonzero(cl)[0].tolist()) <= set(cus)
        assert cl.sum() == tiles
        got = to_host(d_col)
        assert (got[:n] == ref).all() and (got[n:] == 0xEE).all()
        assert (to_host(d_hist).astype(np.uint64) == ref_hist).all()
    # the gate's fallback (no workgroup resident on an allowed CU) is legal
    assert ctx.device_error() & ~sg.DEVFLAG_GATE_FALLBACK == 0


def test_out_of_range_page_entry_is_flagged_not_accessed(ctx):
    shift = 16
    pages = 8
    pt = torch.arange(pages, dtype=torch.int32, device=DEV)
    bad = pt.clone()
    bad[3] = pages + 100
    src = torch.ones(pages * 65536, dtype=torch.uint8, device=DEV)
    dst = torch.zeros_like(src)
    sg.bimodal_relayout(ctx, sg.paged(dst, pt, pages), sg.paged(src, bad, pages),
                        pages * 65536, shift)
    assert ctx.device_error() & sg.DEVERR_PT_RANGE
    d = to_host(dst).reshape(pages, 65536)
    assert (d[3] == 0).all() and (d[[0, 1, 2, 4, 5, 6, 7]] == 1).all()
    assert ctx.device_error() == 0


@pytest.mark.parametrize("shift,B", [(21, 1), (21, 8), (12, 1), (12, 8)])
def test_gemv_out_of_range_page_entry_is_flagged_not_accessed(ctx, orc, shift, B):
    """A W page-table entry beyond the pool: the GEMV reads none of that
    page (its bytes count as zero), raises the range flag, and every output
    equals the oracle's on a copy of W with that page zeroed.  With 2 MiB
    pages every tile lies inside one page (on the MFMA path: a buffer
    resource per row, of length zero for the bad page); with 4 KiB pages a
    tile spans many (a table read per load).  Batch 1 takes the vector
    path, batch 8 the MFMA path."""
    M, K, wd = 1024, 4096, sg.BF16
    say(f"gemv bad page entry: {1 << (shift - 10)} KiB pages, B={B}")
    pool, pt, d_pool, d_pt, pool_pages = upload_w(orc, M, K, wd, shift, range(48), M + B, 1, 6)
    n_pages = -(-M * K * 2 // (1 << shift))
    k = n_pages // 2
    bad = d_pt.clone()
    bad[k] = pool_pages + 100
    xb = x_bits(wd, B * K, 11)
    assert ctx.device_error() == 0
    y = launch_gemv(ctx, d_pool, bad, pool_pages, M, K, B, wd, wd, to_dev(xb), shift, None)
    assert ctx.device_error() == sg.DEVERR_PT_RANGE
    zeroed = pool.copy()
    zeroed.reshape(pool_pages, 1 << shift)[int(pt[k])] = 0
    ref, absdot = orc.gemv(zeroed, pt, wd, M, K, xb, wd, B, shift)
    gemv_check(ctx, y, ref, absdot, M, K, B, wd, wd, None, tag="bad page")


def test_two_streams_disjoint_masks_run_concurrently(ctx, orc):
    """A GEMV stream on CUs 0..3/4 and a triad stream on the rest, launched
    back to back so that they overlap; both results match the oracle and no
    range needed the last-workgroup fallback (the fixture checks the flags)."""
    n = ctx.num_cus
    s_ls, s_be = torch.cuda.Stream(), torch.cuda.Stream()
    sg.set_cu_mask(ctx, s_ls, range(3 * n // 4))
    sg.set_cu_mask(ctx, s_be, range(3 * n // 4, n))
    sg.set_stream_occupancy(ctx, s_be, 3)
    # triad operands: 64 MiB arrays, identity pages
    shift, elems = 16, 1 << 24
    pages = elems * 4 >> shift
    pt = torch.arange(pages, dtype=torch.int32, device=DEV)
    b = synth.uniform_f32(elems, seed=31)
    c = synth.uniform_f32(elems, seed=32)
    d_b, d_c = to_dev(b), to_dev(c)
    d_a = torch.zeros_like(d_b)
    # GEMV operands: bf16 1024x4096 in 64 KiB pages
    M, K = 1024, 4096
    wb = synth.normal_bf16(M * K, seed=33, sigma=0.02)
    xb = synth.normal_bf16(K, seed=34)
    wpages = M * K * 2 >> shift
    wpt = torch.arange(wpages, dtype=torch.int32, device=DEV)
    d_w, d_x = to_dev(wb), to_dev(xb)
    d_y = torch.zeros(M, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    for i in range(4):
        sg.colored_stream(ctx, sg.paged(d_a, pt, pages), sg.paged(d_b, pt, pages),
                          sg.paged(d_c, pt, pages), 3.0, elems, shift, s_be)
        for _ in range(20):
            sg.colored_gemv(ctx, sg.paged(d_w, wpt, wpages), sg.BF16, M, K, d_x, sg.BF16, 1, d_y,
                            shift, s_ls)
    torch.cuda.synchronize()
    sg.set_cu_mask(ctx, s_ls, None)
    sg.set_cu_mask(ctx, s_be, None)
    sg.set_stream_occupancy(ctx, s_be, 0)
    ident = np.arange(pages, dtype=np.uint32)
    ref_a = np.zeros_like(b)
    orc.triad(ref_a, ident, b, ident, c, ident, 3.0, elems, shift)
    assert (to_host(d_a).view(np.uint32) == ref_a.view(np.uint32)).all()
    y_ref, absdot = orc.gemv(wb, np.arange(wpages, dtype=np.uint32), orc.BF16, M, K, xb, orc.BF16,
                             1, shift)
    gemv_ok(to_host(d_y).reshape(1, M), y_ref, absdot)


def test_corun_disjoint_colours_and_cus(ctx, orc):
    """The co-located pair at its real size, from one pool under one hash
    (6 masks on address bits 21..40): the LS GEMV (bf16 4096 x 11008, batch
    1) on colours 0..47 in 2 MiB pages and CUs 0..191, concurrent with the BE
    triad on three 2 GiB fp32 arrays on colours 48..63 in 64 KiB pages and
    CUs 192..255.  The two page sets share no 2 MiB region of the pool; every
    GEMV output is within the oracle bound and 2^18 sampled triad elements
    equal the oracle's fmaf."""
    n_cus = ctx.num_cus
    ls_cus, be_cus = range(n_cus * 3 // 4), range(n_cus * 3 // 4, n_cus)
    masks = synth.xor_masks(6, seed=1, min_bit=21)
    M, K, wshift, shift = 4096, 11008, 21, 16
    elems = 1 << 29
    pages = elems * 4 >> shift
    region = 1 << (wshift - shift)                 # 64 KiB pages per 2 MiB region
    w_pages = -(-(M * K * 2) >> wshift)
    pool_regions = int((3 * pages / region) * 4 * 1.1) + 4 * w_pages + 64
    raw, base, off = aligned_pool(pool_regions, wshift)
    say(f"corun: one pool of {pool_regions} x 2 MiB, masks {[hex(m) for m in masks]}")
    # LS table (2 MiB pages) and BE table (64 KiB pages) from the same pool
    d_wpt = torch.empty(w_pages, dtype=torch.int32, device=DEV)
    sg.colour_alloc_pagetable(ctx, masks, base, wshift, pool_regions, range(48), w_pages, d_wpt)
    d_bpt = torch.empty(3 * pages, dtype=torch.int32, device=DEV)
    sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_regions * region, range(48, 64),
                              3 * pages, d_bpt)
    wpt = to_host(d_wpt).view(np.uint32)
    bpt = to_host(d_bpt).view(np.uint32)
    ref_wpt, _ = orc.pagetable(masks, base, wshift, pool_regions, synth.colour_set_bits(range(48)),
                               w_pages)
    assert (wpt == ref_wpt).all()
    assert not set(wpt.tolist()) & set((bpt // region).tolist())
    # LS weights and BE inputs placed through the tables
    wb = w_bits(sg.BF16, M * K, 41)
    xb = x_bits(sg.BF16, K, 42)
    d_w = to_dev(wb)
    w_ident = torch.arange(w_pages, dtype=torch.int32, device=DEV)
    W = sg.paged(base, d_wpt, pool_regions)
    sg.bimodal_relayout(ctx, W, sg.paged(d_w, w_ident, w_pages), M * K * 2, wshift)
    b = synth.uniform_f32(elems, seed=43)
    c = synth.uniform_f32(elems, seed=44)
    ident = torch.arange(pages, dtype=torch.int32, device=DEV)
    T = [sg.paged(base, d_bpt[i * pages:(i + 1) * pages], pool_regions * region) for i in range(3)]
    for i, h in ((1, b), (2, c)):
        d_h = to_dev(h)
        sg.bimodal_relayout(ctx, T[i], sg.paged(d_h, ident, pages), elems * 4, shift)
        del d_h
    d_x = to_dev(xb)
    d_y = torch.full((M,), float("nan"), dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    s_ls, s_be = torch.cuda.Stream(), torch.cuda.Stream()
    sg.set_cu_mask(ctx, s_ls, ls_cus)
    sg.set_cu_mask(ctx, s_be, be_cus)
    try:
        say("  BE triad 3 x 2 GiB on 64 CUs with 40 LS GEMVs on 192 CUs")
        sg.colored_stream(ctx, T[0], T[1], T[2], 3.0, elems, shift, s_be)
        for _ in range(40):
            sg.colored_gemv(ctx, W, sg.BF16, M, K, d_x, sg.BF16, 1, d_y, wshift, s_ls)
        torch.cuda.synchronize()
    finally:
        sg.set_cu_mask(ctx, s_ls, None)
        sg.set_cu_mask(ctx, s_be, None)
    y_ref, absdot = orc.gemv(wb, np.arange(w_pages, dtype=np.uint32), orc.BF16, M, K, xb,
                             orc.BF16, 1, wshift)
    gemv_check(ctx, to_host(d_y).reshape(1, M), y_ref, absdot, M, K, 1, sg.BF16, sg.BF16,
               ls_cus, tag="c4")
    rng = np.random.default_rng(45)
    idx = np.sort(rng.choice(elems, size=1 << 18, replace=False)).astype(np.int64)
    epp = (1 << shift) // 4
    pa = bpt[:pages].astype(np.int64)
    where = off // 4 + pa[idx // epp] * epp + idx % epp
    got = to_host(raw.view(torch.float32)[torch.from_numpy(where).to(DEV)])
    ref = np.empty(idx.size, np.float32)
    ident_h = np.arange(-(-idx.size // epp), dtype=np.uint32)
    bs = np.zeros(ident_h.size * epp, np.float32); bs[:idx.size] = b[idx]
    cs = np.zeros(ident_h.size * epp, np.float32); cs[:idx.size] = c[idx]
    full = np.zeros(ident_h.size * epp, np.float32)
    orc.triad(full, ident_h, bs, ident_h, cs, ident_h, 3.0, idx.size, shift)
    ref[:] = full[:idx.size]
    assert (got.view(np.uint32) == ref.view(np.uint32)).all()


def test_zz_no_device_flags_raised():
    assert not FLAGS, f"device flags raised (2 = last-workgroup fallback): {FLAGS}"
