"""HIP graph capture of the path.  A classify with histogram and a batch-1
and batch-8 GEMV (static schedule; the classify's finishing kernel is part
of the capture), the allocation-free page-table build, and a triad and a
relayout (ticket queues) are captured once with torch.cuda.graph and the
graph is replayed several times, with the outputs overwritten and other
eager launches in between.  Every replay must equal the eager run bit for
bit, and the eager run must equal the oracle (GEMV: within the bound of its
summation tree).  None of these entry points records a memset or waits on
the host, which is what makes them capturable."""
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
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = sg.Context(0)
    yield c
    c.close()


def dev(a: np.ndarray):
    a = np.ascontiguousarray(a)
    signed = {np.dtype(np.uint8): np.int8, np.dtype(np.uint16): np.int16,
              np.dtype(np.uint32): np.int32, np.dtype(np.uint64): np.int64}
    if a.dtype in signed:
        a = a.view(signed[a.dtype])
    return torch.from_numpy(a).to(DEV)


class Work:
    """Inputs of every captured call and one set of output buffers."""

    def __init__(self):
        rng = np.random.default_rng(7)
        # classify: several wave tiles and a ragged tail
        self.masks = synth.xor_masks(6, seed=1, min_bit=12)
        self.addrs = synth.page_addresses(5 * 1024 + 13, seed=3)
        self.d_addrs = dev(self.addrs)
        # page table: 64 KiB pages of a 50,000-page pool, colours 0..7 of 64
        self.pt_masks = synth.xor_masks(6, seed=1, min_bit=16)
        self.pt_args = (1 << 40, 16, 50000, range(8), 3000)
        # triad and relayout: 64 KiB pages in permuted order
        self.shift = 16
        self.n = 5 * 16384 + 7
        self.pages = 6
        self.pts = [rng.permutation(8)[:self.pages].astype(np.uint32) for _ in range(3)]
        self.b = synth.uniform_f32(8 * 16384, seed=2)
        self.c = synth.uniform_f32(8 * 16384, seed=3)
        self.d_b, self.d_c = dev(self.b), dev(self.c)
        self.d_pts = [dev(p) for p in self.pts]
        self.rel_bytes = self.pages * 65536 - 10
        self.rel_src = synth.random_u16(8 * 32768, seed=4)
        self.d_rel_src = dev(self.rel_src)
        # GEMV: bf16 W [96 x 1024] over permuted 64 KiB pages, batches 1 and 8
        self.M, self.K = 96, 1024
        w_pages = -(-self.M * self.K * 2 // 65536)
        self.w_pt = rng.permutation(w_pages + 2)[:w_pages].astype(np.uint32)
        self.w_pool = synth.normal_bf16((w_pages + 2) * 32768, seed=5, sigma=0.02)
        self.x = synth.normal_bf16(8 * self.K, seed=6)
        self.d_w_pool, self.d_w_pt, self.d_x = dev(self.w_pool), dev(self.w_pt), dev(self.x)
        self.w_pool_pages = w_pages + 2

    def outputs(self):
        return {"colours": torch.empty(self.addrs.size, dtype=torch.uint8, device=DEV),
                "hist": torch.empty(64, dtype=torch.int64, device=DEV),
                "pt": torch.empty(self.pt_args[4], dtype=torch.int32, device=DEV),
                "pt_n": torch.empty(1, dtype=torch.int64, device=DEV),
                "a": torch.empty(8 * 16384, dtype=torch.float32, device=DEV),
                "rel": torch.empty(8 * 32768, dtype=torch.int16, device=DEV),
                "y1": torch.empty(self.M, dtype=torch.float32, device=DEV),
                "y8": torch.empty(8 * self.M, dtype=torch.float32, device=DEV)}

    def run(self, ctx, o):
        """Enqueues every call on the current stream."""
        sg.colour_classify(ctx, self.masks, self.d_addrs, o["colours"], o["hist"])
        origin, shift, pool, S, n = self.pt_args
        sg.colour_alloc_pagetable_noalloc(ctx, self.pt_masks, origin, shift, pool, S, n, o["pt"],
                                          o["pt_n"])
        sg.colored_stream(ctx, sg.paged(o["a"], self.d_pts[0], 8), sg.paged(self.d_b, self.d_pts[1], 8),
                          sg.paged(self.d_c, self.d_pts[2], 8), 3.0, self.n, self.shift)
        sg.bimodal_relayout(ctx, sg.paged(o["rel"], self.d_pts[0], 8),
                            sg.paged(self.d_rel_src, self.d_pts[1], 8), self.rel_bytes, self.shift)
        w = sg.paged(self.d_w_pool, self.d_w_pt, self.w_pool_pages)
        sg.colored_gemv(ctx, w, sg.BF16, self.M, self.K, self.d_x, sg.BF16, 1, o["y1"], 16)
        sg.colored_gemv(ctx, w, sg.BF16, self.M, self.K, self.d_x, sg.BF16, 8, o["y8"], 16)


def fill(o):
    """Overwrite every output with a pattern (fill kernels, not memsets):
    0x5A in the colour bytes, -1 everywhere else."""
    for k, t in o.items():
        t.fill_(0x5A if k == "colours" else -1)


def snapshot(o):
    torch.cuda.synchronize()
    return {k: v.cpu().numpy().copy() for k, v in o.items()}


def check_against_oracle(orc, wk, got):
    cols, hist = orc.classify(wk.addrs, wk.masks)
    assert (got["colours"] == cols).all()
    assert (got["hist"].view(np.uint64) == hist).all()
    origin, shift, pool, S, n = wk.pt_args
    pt, found = orc.pagetable(wk.pt_masks, origin, shift, pool, synth.colour_set_bits(S), n)
    assert int(got["pt_n"][0]) == found >= n
    assert (got["pt"].view(np.uint32) == pt).all()
    a = np.full(8 * 16384, -1.0, dtype=np.float32)   # the pattern the eager run started from
    orc.triad(a, wk.pts[0], wk.b, wk.pts[1], wk.c, wk.pts[2], 3.0, wk.n, wk.shift)
    assert (got["a"].view(np.uint32) == a.view(np.uint32)).all()
    rel = np.full(8 * 32768, -1, dtype=np.int16)
    orc.relayout(rel, wk.pts[0], wk.rel_src, wk.pts[1], wk.rel_bytes, wk.shift)
    assert (got["rel"] == rel).all()
    for B, key in ((1, "y1"), (8, "y8")):
        ref, absdot = orc.gemv(wk.w_pool, wk.w_pt, sg.BF16, wk.M, wk.K, wk.x, sg.BF16, B, 16)
        depth = sg.gemv_plan(256, sg.BF16, wk.M, wk.K, sg.BF16, B)["sum_depth"]
        err = np.abs(got[key].reshape(B, wk.M).astype(np.float64) - ref)
        assert np.all(err <= 2 * depth * 2.0 ** -24 * absdot + 1e-30)


def test_graph_replays_match_eager_and_oracle(ctx, orc):
    wk = Work()
    eager_out, graph_out = wk.outputs(), wk.outputs()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        fill(eager_out)
        for _ in range(2):       # warm-up: kernels loaded, occupancy cached
            wk.run(ctx, eager_out)
        fill(eager_out)
        wk.run(ctx, eager_out)
    eager = snapshot(eager_out)
    say("graph: eager run against the oracle")
    check_against_oracle(orc, wk, eager)

    g = torch.cuda.CUDAGraph()
    fill(graph_out)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        capture_stream = torch.cuda.current_stream().cuda_stream
        wk.run(ctx, graph_out)
    torch.cuda.synchronize()
    other_y = torch.empty(8 * wk.M, dtype=torch.float32, device=DEV)
    w = sg.paged(wk.d_w_pool, wk.d_w_pt, wk.w_pool_pages)
    for r in range(5):
        say(f"graph: replay {r}")
        fill(graph_out)
        g.replay()
        got = snapshot(graph_out)
        for k in eager:
            assert got[k].tobytes() == eager[k].tobytes(), (r, k)
        # eager launches of the same kernels between replays
        with torch.cuda.stream(s):
            sg.colored_gemv(ctx, w, sg.BF16, wk.M, wk.K, wk.d_x, sg.BF16, 8, other_y, 16)
            sg.colour_classify(ctx, wk.masks, wk.d_addrs, eager_out["colours"], eager_out["hist"])
        torch.cuda.synchronize()
        assert other_y.cpu().numpy().tobytes() == eager["y8"].tobytes()
    assert ctx.device_error() == 0
    del g
    torch.cuda.synchronize()
    sg.stream_release(ctx, capture_stream)
    sg.stream_release(ctx, s)
