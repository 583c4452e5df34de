"""Seeded random parity sweep.  Shapes, lengths, page sizes, colour sets,
CU masks and (for the GEMV) batch and dtypes are drawn from fixed seeds;
every case runs one entry point and compares it with the oracle: bit-exact
for classify, histogram, triad and relayout, the summation-tree bound for
the GEMV.  Masks are all CUs, whole XCDs (the static schedule) or a random
subset (the ticket queues)."""
import sys

import numpy as np
import pytest

import synth
import paper_2407_13996_amd as sg
import test_gpu_parity as tp

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = sg.Context(0)
    yield c
    assert c.device_error() == 0
    c.close()


def draw_mask(rng, num_cus):
    """None, whole XCDs or a random subset, one third each."""
    kind = int(rng.integers(0, 3))
    if kind == 0:
        return None
    if kind == 1:
        return range(32 * int(rng.integers(1, num_cus // 32 + 1)))
    return synth.random_cu_subset(num_cus, int(rng.integers(1, num_cus)), seed=int(rng.integers(1 << 30)))


class Masked:
    """Applies a CU mask to the current stream for the duration."""

    def __init__(self, ctx, cus):
        self.ctx, self.cus = ctx, cus

    def __enter__(self):
        if self.cus is not None:
            sg.set_cu_mask(self.ctx, None, self.cus)

    def __exit__(self, *exc):
        if self.cus is not None:
            sg.set_cu_mask(self.ctx, None, None)


def mask_name(cus):
    return "all" if cus is None else f"{len(list(cus))} CUs"


@pytest.mark.parametrize("seed", range(12))
def test_random_classify(ctx, orc, seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(0, 300_000))
    K = int(rng.integers(1, 9))
    hist = bool(rng.integers(0, 2))
    cus = draw_mask(rng, ctx.num_cus)
    say(f"random classify seed={seed}: n={n} K={K} hist={hist} mask {mask_name(cus)}")
    masks = synth.xor_masks(K, seed=seed + 1, min_bit=12)
    addrs = synth.page_addresses(max(n, 1), seed=seed)[:n]
    d_addrs = tp.to_dev(addrs) if n else torch.empty(0, dtype=torch.int64, device=DEV)
    d_col = torch.full((max(n, 16) + 16,), 0xEE, dtype=torch.uint8, device=DEV)
    d_hist = torch.full((1 << K,), 12345, dtype=torch.int64, device=DEV) if hist else None
    with Masked(ctx, cus):
        sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist)
    got = tp.to_host(d_col)
    ref, ref_hist = orc.classify(addrs, masks)
    assert (got[:n] == ref).all()
    assert (got[n:] == 0xEE).all()
    if hist:
        assert (tp.to_host(d_hist).astype(np.uint64) == ref_hist).all()


@pytest.mark.parametrize("seed", range(16))
def test_random_triad(ctx, orc, seed):
    rng = np.random.default_rng(2000 + seed)
    shift = int(rng.integers(10, 22))
    P = 1 << shift
    n = int(rng.integers(0, min(600_000, 40 * P // 4) + 1))
    s = float(np.float32(rng.uniform(-4, 4)))
    cus = draw_mask(rng, ctx.num_cus)
    sets = [range(c0, c0 + w) for c0, w in
            ((int(rng.integers(0, 48)), int(rng.integers(1, 17))) for _ in range(3))]
    say(f"random triad seed={seed}: shift={shift} n={n} s={s} sets "
        f"{[(r.start, r.stop) for r in sets]} mask {mask_name(cus)}")
    n_pages = max(1, -(-n * 4 // P))
    tabs = [tp.make_tables(orc, shift, n_pages, S, 30 + seed + i) for i, S in enumerate(sets)]
    pools = max(t[1] for t in tabs)
    pts = [t[0] for t in tabs]
    epp = P // 4
    a0 = synth.uniform_f32(pools * epp, seed=seed + 1)
    b = synth.uniform_f32(pools * epp, seed=seed + 2)
    c = synth.uniform_f32(pools * epp, seed=seed + 3)
    d_a, d_b, d_c = tp.to_dev(a0), tp.to_dev(b), tp.to_dev(c)
    with Masked(ctx, cus):
        sg.colored_stream(ctx, sg.paged(d_a, tp.to_dev(pts[0]), pools),
                          sg.paged(d_b, tp.to_dev(pts[1]), pools),
                          sg.paged(d_c, tp.to_dev(pts[2]), pools), s, n, shift)
    ref = a0.copy()
    orc.triad(ref, pts[0], b, pts[1], c, pts[2], s, n, shift)
    assert (tp.to_host(d_a).view(np.uint32) == ref.view(np.uint32)).all()


@pytest.mark.parametrize("seed", range(16))
def test_random_relayout(ctx, orc, seed):
    rng = np.random.default_rng(3000 + seed)
    shift = int(rng.integers(10, 22))
    P = 1 << shift
    n_bytes = int(rng.integers(0, min(3_000_000, 40 * P) + 1))
    cus = draw_mask(rng, ctx.num_cus)
    say(f"random relayout seed={seed}: shift={shift} n_bytes={n_bytes} mask {mask_name(cus)}")
    n_pages = max(1, -(-n_bytes // P))
    pt_s, src_pages = tp.make_tables(orc, shift, n_pages, range(int(rng.integers(0, 32)), 48), 50 + seed)
    pt_d, dst_pages = tp.make_tables(orc, shift, n_pages, range(int(rng.integers(1, 64))), 90 + seed)
    src = synth.random_bytes(src_pages * P, seed=seed + 5)
    dst0 = synth.random_bytes(dst_pages * P, seed=seed + 6)
    d_src, d_dst = tp.to_dev(src), tp.to_dev(dst0)
    with Masked(ctx, cus):
        sg.bimodal_relayout(ctx, sg.paged(d_dst, tp.to_dev(pt_d), dst_pages),
                            sg.paged(d_src, tp.to_dev(pt_s), src_pages), n_bytes, shift)
    ref = dst0.copy()
    orc.relayout(ref, pt_d, src, pt_s, n_bytes, shift)
    assert (tp.to_host(d_dst) == ref).all()


DTYPES = [(sg.BF16, sg.BF16), (sg.F16, sg.F16), (sg.F32, sg.F32), (sg.BF16, sg.F32),
          (sg.F32, sg.BF16), (sg.F16, sg.F32), (sg.F32, sg.F16), (sg.BF16, sg.F16)]
SIZE = {sg.F32: 4, sg.BF16: 2, sg.F16: 2}


@pytest.mark.parametrize("seed", range(48))
def test_random_gemv(ctx, orc, seed):
    rng = np.random.default_rng(4000 + seed)
    wd, xd = DTYPES[int(rng.integers(0, len(DTYPES)))] if seed % 3 else DTYPES[seed % 2]
    B = int(rng.integers(1, 9))
    M = int(rng.integers(1, 1500))
    step = 16 // SIZE[wd]                   # rows are whole 16-byte slices
    K = step * int(rng.integers(1, 6000 // step + 1))
    row = K * SIZE[wd]
    # a tile's rows (16 at most) must span at most 254 pages
    lo = max(10, int(np.ceil(np.log2(max(1, 16 * row / 250)))))
    shift = int(rng.integers(lo, 22))
    cus = draw_mask(rng, ctx.num_cus)
    S = range(int(rng.integers(0, 16)), int(rng.integers(17, 65)))
    say(f"random gemv seed={seed}: {M}x{K} B={B} w={wd} x={xd} shift={shift} colours "
        f"{S.start}..{S.stop - 1} mask {mask_name(cus)}")
    pool, pt, d_pool, d_pt, pool_pages = tp.upload_w(orc, M, K, wd, shift, S, seed, seed + 1, 6)
    xb = tp.x_bits(xd, B * K, seed + 2)
    y = tp.launch_gemv(ctx, d_pool, d_pt, pool_pages, M, K, B, wd, xd, tp.to_dev(xb), shift,
                       tp.cu_list(cus))
    ref, absdot = orc.gemv(pool, pt, wd, M, K, xb, xd, B, shift)
    tp.gemv_check(ctx, y, ref, absdot, M, K, B, wd, xd, tp.cu_list(cus), tag=f"random {seed}")


@pytest.mark.parametrize("seed", range(16))
def test_random_pagetable(ctx, orc, seed):
    """Random hashes (mask bits up to three positions inside the page, so a
    page may carry several colours), pool sizes, origins, colour sets and
    table lengths, through the synchronous and the allocation-free builds;
    a shortfall must report the oracle's count."""
    rng = np.random.default_rng(5000 + seed)
    shift = int(rng.integers(10, 22))
    K = int(rng.integers(1, 9))
    lo = int(rng.integers(max(8, shift - 3), shift + 5))
    masks = synth.xor_masks(K, seed=seed + 7, min_bit=lo)
    pool = int(rng.integers(1, 200_001))
    origin = int(rng.integers(0, 1 << (40 - shift))) << shift
    S = sorted(int(c) for c in rng.choice(1 << K, size=int(rng.integers(1, (1 << K) + 1)),
                                        replace=False))
    n = int(rng.integers(1, pool + 1))
    cus = draw_mask(rng, ctx.num_cus)
    say(f"random pagetable seed={seed}: shift={shift} K={K} mask bits from {lo} pool={pool} "
        f"|S|={len(S)} n={n} mask {mask_name(cus)}")
    ref, ref_found = orc.pagetable(masks, origin, shift, pool, synth.colour_set_bits(S), n)
    d_pt = torch.full((n + 8,), -1, dtype=torch.int32, device=DEV)
    with Masked(ctx, cus):
        if ref_found >= n:
            assert sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, n, d_pt) == ref_found
        else:
            with pytest.raises(sg.SgdrcError) as e:
                sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, n, d_pt)
            assert e.value.code == sg.ENOMEM and e.value.n_found == ref_found
    k = min(n, ref_found)
    got = tp.to_host(d_pt).view(np.uint32)
    assert (got[:k] == ref[:k]).all()
    assert (got[n:] == 0xFFFFFFFF).all()
    # the allocation-free build writes the same table and the full count
    d_pt2 = torch.full((n + 8,), -1, dtype=torch.int32, device=DEV)
    d_found = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    with Masked(ctx, cus):
        sg.colour_alloc_pagetable_noalloc(ctx, masks, origin, shift, pool, S, n, d_pt2, d_found)
    assert int(tp.to_host(d_found)[0]) == ref_found
    assert (tp.to_host(d_pt2).view(np.uint32)[:k] == ref[:k]).all()


@pytest.mark.parametrize("seed", range(8))
def test_random_colour_table(ctx, orc, seed):
    """Colour tables (paper section 5.3) of random size, partition size,
    origin and holes: classify (with or without the 256-bin histogram,
    addresses inside, below and past the table) and the page-table build
    (pages of 1 KiB to 64 KiB, pools reaching past either end of the table)
    against the oracle."""
    rng = np.random.default_rng(6000 + seed)
    lut_shift = int(rng.integers(10, 14))
    entries = int(rng.integers(1, 1 << 17))
    origin = int(rng.integers(1, 1 << 20)) << 20
    lut = tp.random_table(entries, seed=seed, colours=int(rng.integers(1, 257)) if seed % 2 else 64,
                          holes=float(rng.uniform(0, 0.05)))
    t = sg.colour_table(tp.to_dev(lut), origin, lut_shift)
    cus = draw_mask(rng, ctx.num_cus)
    n = int(rng.integers(0, 200_000))
    hist = bool(rng.integers(0, 2))
    span = entries << lut_shift
    addrs = (origin + rng.integers(-(1 << 16), span + (1 << 16), size=max(n, 1))).astype(np.uint64)[:n]
    say(f"random colour table seed={seed}: {entries} partitions of 2^{lut_shift}, n={n} "
        f"hist={hist} mask {mask_name(cus)}")
    d_addrs = tp.to_dev(addrs) if n else torch.empty(0, dtype=torch.int64, device=DEV)
    d_col = torch.full((max(n, 16) + 16,), 0xEE, dtype=torch.uint8, device=DEV)
    d_hist = torch.full((256,), 777, dtype=torch.int64, device=DEV) if hist else None
    with Masked(ctx, cus):
        sg.colour_classify_table(ctx, t, d_addrs, d_col, d_hist)
    ref, ref_hist = orc.classify_lut(addrs, lut, origin, lut_shift)
    got = tp.to_host(d_col)
    assert (got[:n] == ref).all() and (got[n:] == 0xEE).all()
    if hist:
        assert (tp.to_host(d_hist).astype(np.uint64) == ref_hist).all()
    # page tables through the same table
    page_shift = int(rng.integers(10, 17))
    addr_origin = (origin - (int(rng.integers(0, 64)) << page_shift))
    pool = max(1, (span + int(rng.integers(0, 1 << 17))) >> page_shift)
    # colours 0..254 (255 marks a partition with no colour)
    S = sorted(int(c) for c in rng.choice(255, size=int(rng.integers(1, 256)), replace=False))
    ref_pt, ref_found = orc.pagetable_lut(lut, origin, lut_shift, addr_origin, page_shift, pool,
                                          synth.colour_set_bits(S), pool)
    n_need = int(rng.integers(1, pool + 1))
    say(f"  table page tables: pages 2^{page_shift}, pool {pool}, |S|={len(S)}, need {n_need}, "
        f"oracle finds {ref_found}")
    d_pt = torch.full((n_need + 8,), -1, dtype=torch.int32, device=DEV)
    with Masked(ctx, cus):
        if ref_found >= n_need:
            assert sg.colour_alloc_pagetable_table(ctx, t, addr_origin, page_shift, pool, S, n_need,
                                                   d_pt) == ref_found
        else:
            with pytest.raises(sg.SgdrcError) as e:
                sg.colour_alloc_pagetable_table(ctx, t, addr_origin, page_shift, pool, S, n_need,
                                                d_pt)
            assert e.value.code == sg.ENOMEM and e.value.n_found == ref_found
    k = min(n_need, ref_found)
    got = tp.to_host(d_pt).view(np.uint32)
    assert (got[:k] == ref_pt[:k]).all() and (got[n_need:] == 0xFFFFFFFF).all()


@pytest.mark.parametrize("seed", range(6))
def test_random_relayout_batch(ctx, orc, seed):
    """Batches of 1 to 40 relayout items of random page sizes (1 to 64 KiB)
    and lengths (empty ones included) under random CU masks."""
    rng = np.random.default_rng(7000 + seed)
    n_items = int(rng.integers(1, 41))
    cus = draw_mask(rng, ctx.num_cus)
    say(f"random relayout batch seed={seed}: {n_items} items, mask {mask_name(cus)}")
    items, refs, devs, keep = [], [], [], []
    for i in range(n_items):
        shift = int(rng.integers(10, 17))   # 2 MiB pages: in the single relayout sweep
        P = 1 << shift
        n_bytes = 0 if rng.random() < 0.1 else int(rng.integers(1, min(400_000, 8 * P) + 1))
        n_pages = max(1, -(-n_bytes // P))
        pt_s, src_pages = tp.make_tables(orc, shift, n_pages, range(16), 300 + 40 * seed + i)
        pt_d, dst_pages = tp.make_tables(orc, shift, n_pages, range(32, 48), 700 + 40 * seed + i)
        src = synth.random_bytes(src_pages * P, seed=1000 * seed + i)
        dst0 = synth.random_bytes(dst_pages * P, seed=1000 * seed + 500 + i)
        d_src, d_dst, d_ps, d_pd = tp.to_dev(src), tp.to_dev(dst0), tp.to_dev(pt_s), tp.to_dev(pt_d)
        keep += [d_src, d_ps, d_pd]
        items.append((sg.paged(d_dst, d_pd, dst_pages), sg.paged(d_src, d_ps, src_pages), n_bytes,
                      shift))
        ref = dst0.copy()
        orc.relayout(ref, pt_d, src, pt_s, n_bytes, shift)
        refs.append(ref)
        devs.append(d_dst)
    with Masked(ctx, cus):
        sg.bimodal_relayout_batch(ctx, items)
    for i, (d, ref) in enumerate(zip(devs, refs)):
        assert (tp.to_host(d) == ref).all(), i


@pytest.mark.parametrize("seed", range(6))
def test_random_preemption(ctx, orc, seed):
    """A preemptible triad evicted at a random tile (the eviction hook), its
    resumption evicted again at a later random tile or not, then finished,
    each launch under a random CU mask: every tile worked exactly once and
    the result equals the oracle's."""
    import test_gpu_preempt as tpp
    rng = np.random.default_rng(8000 + seed)
    n = int(rng.integers(1, 16 * 1024 * 1024))
    tr = tpp.Triad(orc, 16, n, seed=90 + seed)
    h1 = int(rng.integers(1, tr.tiles + 2))
    h2 = int(rng.integers(h1 + 1, tr.tiles + 3)) if rng.random() < 0.6 else 0
    masks = [draw_mask(rng, ctx.num_cus) for _ in range(3)]
    say(f"random preemption seed={seed}: n={n} ({tr.tiles} tiles), evicted at {h1}, then "
        f"{h2 or 'not'}; masks {[mask_name(m) for m in masks]}")
    st = torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    logs = tpp.Logs(ctx, tr.tiles)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        sg.set_cu_mask(ctx, st, masks[0])
        sg.set_eviction_hook(ctx, st, h1)
        tr.launch(ctx, st)
        left1 = sg.suspended(ctx, st)
        if h2:
            sg.set_cu_mask(ctx, st, masks[1])
            sg.set_eviction_hook(ctx, st, h2)
            sg.resume(ctx, st)
        left2 = sg.suspended(ctx, st)
        say(f"  left after the first launch {left1}, after the second {left2}")
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, masks[2])
        tpp.finish(ctx, st)
        cl, tl = logs.snapshot()
    finally:
        logs.close()
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, None)
        sg.set_eviction_flag(ctx, st, None)
        sg.stream_release(ctx, st)
    tr.check()
    assert (tl == 1).all(), np.unique(tl, return_counts=True)
    assert cl.sum() == tr.tiles
