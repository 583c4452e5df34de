"""Preemptible best-effort launches (paper section 7.1) on the GPU: an
eviction flag stops a persistent triad or relayout at a tile boundary, the
launch ends suspended, and sgdrc_resume finishes it under another CU mask.
The interrupted and resumed launches together must equal one uninterrupted
launch (the oracle's result, bit for bit), with every tile processed
exactly once and the resumed tiles only on the new mask's CUs."""
import sys

import numpy as np
import pytest

import synth
import paper_2407_13996_amd as sg

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def ctx(orc):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = sg.Context(0)
    yield c
    c.close()


@pytest.fixture(autouse=True)
def no_device_flags(ctx):
    ctx.device_error()
    yield
    assert ctx.device_error() == 0


def to_dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    elif a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(DEV)


def to_host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


class Triad:
    """Three coloured arrays of n fp32 elements (oracle page tables) and the
    oracle's a = b + 3 c."""

    def __init__(self, orc, shift, n, seed):
        P = 1 << shift
        self.shift, self.n = shift, n
        n_pages = -(-n * 4 // P)
        self.pools = int(n_pages * 64 / 16 * 1.5) + 64
        self.pts = []
        for i in range(3):
            masks = synth.xor_masks(6, seed=seed + i, min_bit=shift)
            pt, found = orc.pagetable(masks, 0, shift, self.pools,
                                      synth.colour_set_bits(range(8 * i, 8 * i + 16)), n_pages)
            assert found >= n_pages
            self.pts.append(pt)
        epp = P // 4
        self.a0 = synth.uniform_f32(self.pools * epp, seed=seed + 5)
        b = synth.uniform_f32(self.pools * epp, seed=seed + 6)
        c = synth.uniform_f32(self.pools * epp, seed=seed + 7)
        self.d_a, self.d_b, self.d_c = to_dev(self.a0), to_dev(b), to_dev(c)
        self.ref = self.a0.copy()
        orc.triad(self.ref, self.pts[0], b, self.pts[1], c, self.pts[2], 3.0, n, shift)
        self.tiles = -(-(n * 4 & ~15) // 65536)

    def reset(self):
        self.d_a.copy_(to_dev(self.a0))
        torch.cuda.synchronize()

    def launch(self, ctx, stream):
        d_pts = [to_dev(p) for p in self.pts]
        self._keep = d_pts
        sg.colored_stream(ctx, sg.paged(self.d_a, d_pts[0], self.pools),
                          sg.paged(self.d_b, d_pts[1], self.pools),
                          sg.paged(self.d_c, d_pts[2], self.pools), 3.0, self.n, self.shift,
                          stream)

    def check(self):
        assert (to_host(self.d_a).view(np.uint32) == self.ref.view(np.uint32)).all()


class Logs:
    def __init__(self, ctx, n_tiles):
        self.ctx = ctx
        self.cu = torch.zeros(ctx.num_cus, dtype=torch.int32, device=DEV)
        self.tile = torch.zeros(max(n_tiles, 1), dtype=torch.int32, device=DEV)
        ctx.set_worklog(self.cu, self.tile)

    def snapshot(self):
        return to_host(self.cu).copy(), to_host(self.tile).copy()

    def close(self):
        self.ctx.set_worklog(None, None)


def test_triad_evicted_before_start_resumes_on_other_cus(ctx, orc):
    n_cu = ctx.num_cus
    tr = Triad(orc, 16, 600 * 16384 + 7, seed=40)
    st = torch.cuda.Stream()
    flag = torch.ones(1, dtype=torch.int32, device=DEV)
    logs = Logs(ctx, tr.tiles)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        tr.launch(ctx, st)
        left = sg.suspended(ctx, st)
        say(f"evicted before start: {left} of {tr.tiles} tiles left")
        assert left == tr.tiles
        assert (to_host(tr.d_a).view(np.uint32) == tr.a0.view(np.uint32)).all()
        cl, tl = logs.snapshot()
        assert tl.sum() == 0
        flag.zero_()
        torch.cuda.synchronize()
        sg.set_cu_mask(ctx, st, range(n_cu // 2, n_cu))
        sg.resume(ctx, st)
        assert sg.suspended(ctx, st) == 0
        cl, tl = logs.snapshot()
    finally:
        logs.close()
        sg.set_cu_mask(ctx, st, None)
        sg.set_eviction_flag(ctx, st, None)
    tr.check()
    assert (tl == 1).all()
    assert set(np.nonzero(cl)[0].tolist()) <= set(range(n_cu // 2, n_cu))


def _delay(stream, us):
    """Enqueue on ``stream`` work that takes roughly ``us`` microseconds."""
    with torch.cuda.stream(stream):
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(int(us * 100))
        else:
            x = torch.empty(int(us * 2e5), device=DEV)
            x.normal_()


def finish(ctx, st, rounds=4):
    """Resume ``st`` until its preemptible launch has no tiles left."""
    r = 0
    while sg.suspended(ctx, st) and r < rounds:
        sg.resume(ctx, st)
        r += 1
    assert sg.suspended(ctx, st) == 0


@pytest.mark.parametrize("at", [64, 1000, 3000])
def test_triad_evicted_mid_run_every_tile_once(ctx, orc, at):
    """Evicted mid-run at a chosen tile (the eviction hook makes the flag
    count as raised from tile ``at`` on: workgroups past it stop, tickets
    claimed past it are handed back), then resumed on a quarter of the CUs:
    every tile processed once, the result exact."""
    n_cu = ctx.num_cus
    tr = Triad(orc, 16, 64 * 1024 * 1024 + 3, seed=50)    # 256 MiB arrays, 4097 tiles
    st = torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    logs = Logs(ctx, tr.tiles)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        sg.set_eviction_hook(ctx, st, at)
        tr.launch(ctx, st)
        left = sg.suspended(ctx, st)
        say(f"evicted from tile {at}: {left} of {tr.tiles} tiles left")
        assert 0 < left < tr.tiles - at + 1
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, range(n_cu // 4))
        finish(ctx, st)
        cl, tl = logs.snapshot()
    finally:
        logs.close()
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, None)
        sg.set_eviction_flag(ctx, st, None)
    tr.check()
    assert (tl == 1).all(), np.unique(tl, return_counts=True)
    assert cl.sum() == tr.tiles


def test_triad_evicted_by_another_stream(ctx, orc):
    """The flag raised by a kernel on another stream while the triad runs
    (wherever the timing puts it): after resumptions on a smaller mask,
    every tile was processed once and the result is exact."""
    n_cu = ctx.num_cus
    tr = Triad(orc, 16, 64 * 1024 * 1024 + 3, seed=52)
    st, st2 = torch.cuda.Stream(), torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    for delay_us in (5, 40, 160):
        tr.reset()
        flag.zero_()
        torch.cuda.synchronize()
        logs = Logs(ctx, tr.tiles)
        try:
            sg.set_eviction_flag(ctx, st, flag)
            tr.launch(ctx, st)
            _delay(st2, delay_us)
            with torch.cuda.stream(st2):
                flag.fill_(1)
            left = sg.suspended(ctx, st)
            torch.cuda.synchronize()
            say(f"flag after ~{delay_us} us: {left} of {tr.tiles} tiles left")
            flag.zero_()
            torch.cuda.synchronize()
            sg.set_cu_mask(ctx, st, range(n_cu // 4))
            finish(ctx, st)
            cl, tl = logs.snapshot()
        finally:
            logs.close()
            sg.set_cu_mask(ctx, st, None)
            sg.set_eviction_flag(ctx, st, None)
        tr.check()
        assert (tl == 1).all(), np.unique(tl, return_counts=True)
        assert cl.sum() == tr.tiles


def test_triad_resumption_evicted_mid_run_again(ctx, orc):
    """Evicted at tile 1000, resumed on 16 CUs and evicted again at tile
    2500 (the tiles handed back by the first eviction are worked through
    first), then finished on all CUs: every tile once."""
    tr = Triad(orc, 16, 64 * 1024 * 1024 + 3, seed=55)    # 256 MiB arrays, 4097 tiles
    st = torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    logs = Logs(ctx, tr.tiles)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        sg.set_eviction_hook(ctx, st, 1000)
        tr.launch(ctx, st)
        left1 = sg.suspended(ctx, st)
        sg.set_eviction_hook(ctx, st, 2500)
        sg.set_cu_mask(ctx, st, range(16))
        sg.resume(ctx, st)
        left2 = sg.suspended(ctx, st)
        say(f"evicted at tile 1000: {left1} left; resumed on 16 CUs, evicted at 2500: "
            f"{left2} left of {tr.tiles}")
        assert 0 < left2 < left1 < tr.tiles
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, None)
        finish(ctx, st)
        cl, tl = logs.snapshot()
    finally:
        logs.close()
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, None)
        sg.set_eviction_flag(ctx, st, None)
    tr.check()
    assert (tl == 1).all(), np.unique(tl, return_counts=True)
    assert cl.sum() == tr.tiles


def test_resume_after_completion_does_nothing(ctx, orc):
    tr = Triad(orc, 12, 5 * 1024 + 77, seed=60)
    st = torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    logs = Logs(ctx, tr.tiles)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        tr.launch(ctx, st)
        assert sg.suspended(ctx, st) == 0
        sg.resume(ctx, st)
        sg.resume(ctx, st)
        assert sg.suspended(ctx, st) == 0
        cl, tl = logs.snapshot()
    finally:
        logs.close()
        sg.set_eviction_flag(ctx, st, None)
    tr.check()
    assert (tl == 1).all()


def test_evicted_resumption_stays_suspended(ctx, orc):
    tr = Triad(orc, 16, 40 * 16384, seed=70)
    st = torch.cuda.Stream()
    flag = torch.ones(1, dtype=torch.int32, device=DEV)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        tr.launch(ctx, st)
        assert sg.suspended(ctx, st) == tr.tiles
        sg.resume(ctx, st)                      # flag still set: no progress
        assert sg.suspended(ctx, st) == tr.tiles
        flag.zero_()
        torch.cuda.synchronize()
        sg.resume(ctx, st)
        assert sg.suspended(ctx, st) == 0
    finally:
        sg.set_eviction_flag(ctx, st, None)
    tr.check()


def test_fresh_launch_drops_unresumed_suspension(ctx, orc):
    first = Triad(orc, 16, 20 * 16384 + 1, seed=80)
    second = Triad(orc, 16, 30 * 16384 + 2, seed=90)
    st = torch.cuda.Stream()
    flag = torch.ones(1, dtype=torch.int32, device=DEV)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        first.launch(ctx, st)
        assert sg.suspended(ctx, st) == first.tiles
        flag.zero_()
        torch.cuda.synchronize()
        second.launch(ctx, st)                  # discards the first launch's rest
        assert sg.suspended(ctx, st) == 0
    finally:
        sg.set_eviction_flag(ctx, st, None)
    assert ctx.device_error() == sg.DEVERR_SUSPENDED_DROPPED
    second.check()
    assert (to_host(first.d_a).view(np.uint32) == first.a0.view(np.uint32)).all()


@pytest.mark.parametrize("shift,n_bytes", [(16, 64 * 65536 + 17), (12, 37 * 4096 + 1234)])
def test_relayout_evicted_then_resumed(ctx, orc, shift, n_bytes):
    P = 1 << shift
    n_pages = -(-n_bytes // P)
    pool = int(n_pages * 4 * 1.5) + 64
    masks = synth.xor_masks(6, seed=3, min_bit=shift)
    pt_s, f1 = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits(range(16)), n_pages)
    pt_d, f2 = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits(range(16, 32)), n_pages)
    assert min(f1, f2) >= n_pages
    src = synth.random_u16(pool * P // 2, seed=4)
    d_src = to_dev(src)
    d_dst = torch.zeros(pool * P // 2, dtype=torch.int16, device=DEV)
    ref = np.zeros(pool * P, dtype=np.uint8)
    orc.relayout(ref, pt_d, src.view(np.uint8), pt_s, n_bytes, shift)
    st = torch.cuda.Stream()
    flag = torch.ones(1, dtype=torch.int32, device=DEV)
    dpt_s, dpt_d = to_dev(pt_s), to_dev(pt_d)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        sg.bimodal_relayout(ctx, sg.paged(d_dst, dpt_d, pool), sg.paged(d_src, dpt_s, pool),
                            n_bytes, shift, st)
        assert sg.suspended(ctx, st) > 0
        assert (to_host(d_dst) == 0).all()
        flag.zero_()
        torch.cuda.synchronize()
        sg.set_cu_mask(ctx, st, range(0, ctx.num_cus, 3))
        sg.resume(ctx, st)
        assert sg.suspended(ctx, st) == 0
    finally:
        sg.set_cu_mask(ctx, st, None)
        sg.set_eviction_flag(ctx, st, None)
    assert (to_host(d_dst).view(np.uint8) == ref).all()


@pytest.mark.parametrize("at", [100, 1000])
def test_relayout_evicted_mid_run_every_tile_once(ctx, orc, at):
    """A 128 MiB relayout on 16 CUs evicted mid-run at tile ``at`` (tickets
    claimed past it are handed back), then finished on all CUs: byte-exact,
    every 64 KiB tile once."""
    shift, n_bytes = 16, 128 * 1024 * 1024 + 9
    P = 1 << shift
    n_pages = -(-n_bytes // P)
    tiles = -(-(n_bytes & ~15) // 65536)
    pool = int(n_pages * 4 * 1.5) + 64
    masks = synth.xor_masks(6, seed=5, min_bit=shift)
    pt_s, f1 = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits(range(16)), n_pages)
    pt_d, f2 = orc.pagetable(masks, 0, shift, pool, synth.colour_set_bits(range(16, 32)), n_pages)
    assert min(f1, f2) >= n_pages
    src = synth.random_u16(pool * P // 2, seed=6)
    d_src = to_dev(src)
    d_dst = torch.zeros(pool * P // 2, dtype=torch.int16, device=DEV)
    ref = np.zeros(pool * P, dtype=np.uint8)
    orc.relayout(ref, pt_d, src.view(np.uint8), pt_s, n_bytes, shift)
    st = torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    dpt_s, dpt_d = to_dev(pt_s), to_dev(pt_d)
    logs = Logs(ctx, tiles)
    try:
        sg.set_eviction_flag(ctx, st, flag)
        sg.set_eviction_hook(ctx, st, at)
        sg.set_cu_mask(ctx, st, range(16))
        sg.bimodal_relayout(ctx, sg.paged(d_dst, dpt_d, pool), sg.paged(d_src, dpt_s, pool),
                            n_bytes, shift, st)
        left = sg.suspended(ctx, st)
        say(f"relayout evicted from tile {at}: {left} of {tiles} tiles left")
        assert 0 < left < tiles - at + 1
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, None)
        finish(ctx, st)
        cl, tl = logs.snapshot()
    finally:
        logs.close()
        sg.set_eviction_hook(ctx, st, 0)
        sg.set_cu_mask(ctx, st, None)
        sg.set_eviction_flag(ctx, st, None)
    assert (to_host(d_dst).view(np.uint8) == ref).all()
    assert (tl == 1).all(), np.unique(tl, return_counts=True)
    assert cl.sum() == tiles


def test_stream_release_forgets_state_and_returns_queues(ctx, orc):
    """sgdrc_stream_release: 100 preemptible streams in turn (two work
    queues each, 200 in all against 64 per context) each run a triad and
    are released; a released stream handle starts again on all CUs; a
    suspended launch is dropped on release."""
    n_cu = ctx.num_cus
    tr = Triad(orc, 16, 40 * 16384, seed=110)
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    for i in range(100):
        s = torch.cuda.Stream()
        sg.set_eviction_flag(ctx, s, flag)
        sg.set_cu_mask(ctx, s, [i % n_cu])
        tr.launch(ctx, s)
        assert sg.suspended(ctx, s) == 0
        sg.stream_release(ctx, s)
    tr.check()
    st = torch.cuda.Stream()
    sg.set_cu_mask(ctx, st, range(8))
    sg.stream_release(ctx, st)
    logs = Logs(ctx, tr.tiles)
    try:
        tr.reset()
        tr.launch(ctx, st)                      # same handle: all CUs again
        cl, tl = logs.snapshot()
    finally:
        logs.close()
    tr.check()
    assert (tl == 1).all() and len(set(np.nonzero(cl)[0].tolist()) - set(range(8))) > 0
    # a suspended launch is discarded by the release
    flag.fill_(1)
    torch.cuda.synchronize()
    sg.set_eviction_flag(ctx, st, flag)
    tr.launch(ctx, st)
    assert sg.suspended(ctx, st) == tr.tiles
    sg.stream_release(ctx, st)
    assert ctx.device_error() == sg.DEVERR_SUSPENDED_DROPPED
    flag.zero_()
    sg.stream_release(ctx, torch.cuda.Stream())  # never used: nothing to do


def test_tidal_handover_ls_gemv_and_evicted_triad(ctx, orc):
    """The section 7.1 sequence on one GPU: a best-effort triad runs on all
    CUs; a latency-sensitive GEMV arrives, the triad is evicted, the
    sliding-window policy splits the CUs, the GEMV runs on its share while
    the triad resumes on the rest; both results are exact."""
    n_cu = ctx.num_cus
    tr = Triad(orc, 16, 64 * 1024 * 1024, seed=100)
    be, ls = torch.cuda.Stream(), torch.cuda.Stream()
    flag = torch.zeros(1, dtype=torch.int32, device=DEV)
    M, K, B = 1024, 4096, 1
    w = (synth.normal_f32(M * K, seed=9) * 0.02).astype(np.float32)
    x = synth.normal_f32(B * K, seed=10).astype(np.float32)
    wpt = np.arange(-(-M * K * 4 // 65536), dtype=np.uint32)
    d_w, d_x, d_wpt = to_dev(w), to_dev(x), to_dev(wpt)
    d_y = torch.zeros(B * M, dtype=torch.float32, device=DEV)
    ls_cus, be_cus = sg.tidal_masks(n_cu, [40, 96, 64], window=2, granule=32)
    assert len(ls_cus) == 96 and len(be_cus) == n_cu - 96
    stamp = torch.zeros(1, dtype=torch.int64, device=DEV)
    try:
        # all of it enqueued without waiting on the host: LS raises the flag
        # in its own stream order, BE clears it after its evicted kernel and
        # resumes on the CUs that the window leaves it
        sg.set_eviction_flag(ctx, be, flag)
        tr.launch(ctx, be)
        _delay(ls, 20)
        sg.signal_flag(ctx, ls, flag, 1, stamp)
        sg.set_cu_mask(ctx, ls, ls_cus)
        sg.colored_gemv(ctx, sg.paged(d_w, d_wpt, len(wpt)), sg.F32, M, K, d_x, sg.F32, B,
                        d_y, 16, ls)
        sg.signal_flag(ctx, be, flag, 0)
        sg.set_cu_mask(ctx, be, be_cus)
        sg.resume(ctx, be)
        torch.cuda.synchronize()
        assert sg.suspended(ctx, be) == 0
        assert int(to_host(stamp)[0]) > 0
    finally:
        sg.set_cu_mask(ctx, be, None)
        sg.set_cu_mask(ctx, ls, None)
        sg.set_eviction_flag(ctx, be, None)
    tr.check()
    ref, absdot = orc.gemv(w, wpt, sg.F32, M, K, x, sg.F32, B, 16)
    y = to_host(d_y).reshape(B, M).astype(np.float64)
    assert np.all(np.abs(y - ref) <= 1e-3 * absdot + 1e-30)
