"""One context used from several host threads at once (the header allows
it): each thread owns a stream with its own CU mask (two whole XCDs, or a
random subset of CUs) and runs classify, the triad and the GEMV on it in a
loop, then releases the stream.  Every result must equal the oracle's, and
no device flag may be raised."""
import sys
import threading

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
    c.close()


class Job:
    """Inputs and oracle results of one thread's work."""

    def __init__(self, orc, seed):
        rng = np.random.default_rng(seed)
        # classify
        self.K = int(rng.integers(3, 9))
        self.masks = synth.xor_masks(self.K, seed=seed, min_bit=12)
        self.addrs = synth.page_addresses(int(rng.integers(1000, 60000)), seed=seed)
        self.cols, self.hist = orc.classify(self.addrs, self.masks)
        # triad in 64 KiB pages
        self.shift = 16
        self.n = int(rng.integers(1, 400_000))
        n_pages = -(-self.n * 4 // (1 << self.shift))
        tabs = [tp.make_tables(orc, self.shift, n_pages, range(16 * i, 16 * i + 16), seed + i)
                for i in range(3)]
        self.pools = max(t[1] for t in tabs)
        self.pts = [t[0] for t in tabs]
        epp = (1 << self.shift) // 4
        self.a0 = synth.uniform_f32(self.pools * epp, seed=seed + 1)
        self.b = synth.uniform_f32(self.pools * epp, seed=seed + 2)
        self.c = synth.uniform_f32(self.pools * epp, seed=seed + 3)
        self.a_ref = self.a0.copy()
        orc.triad(self.a_ref, self.pts[0], self.b, self.pts[1], self.c, self.pts[2], 2.5, self.n,
                  self.shift)
        # GEMV: bf16, batch 1 or 8
        self.M, self.K_w, self.B = int(rng.integers(50, 800)), 8 * int(rng.integers(16, 400)), \
            int(rng.choice([1, 8]))
        self.w_pool, self.w_pt, _, _, self.w_pool_pages = tp.upload_w(
            orc, self.M, self.K_w, sg.BF16, 16, range(48), seed, seed + 1, 6)
        self.x = tp.x_bits(sg.BF16, self.B * self.K_w, seed + 2)
        self.y_ref, self.absdot = orc.gemv(self.w_pool, self.w_pt, sg.BF16, self.M, self.K_w, self.x,
                                           sg.BF16, self.B, 16)


def worker(ctx, job, cus, rounds, out, idx):
    try:
        st = torch.cuda.Stream()
        with torch.cuda.stream(st):
            d_addrs = tp.to_dev(job.addrs)
            d_col = torch.empty(job.addrs.size, dtype=torch.uint8, device=DEV)
            d_hist = torch.empty(1 << job.K, dtype=torch.int64, device=DEV)
            d_pts = [tp.to_dev(p) for p in job.pts]
            d_b, d_c = tp.to_dev(job.b), tp.to_dev(job.c)
            d_a = tp.to_dev(job.a0)
            w = sg.paged(tp.to_dev(job.w_pool), tp.to_dev(job.w_pt), job.w_pool_pages)
            d_x = tp.to_dev(job.x)
            d_y = torch.empty(job.B * job.M, dtype=torch.float32, device=DEV)
            sg.set_cu_mask(ctx, st, cus)
            for _ in range(rounds):
                sg.colour_classify(ctx, job.masks, d_addrs, d_col, d_hist, st)
                d_a.copy_(tp.to_dev(job.a0))
                sg.colored_stream(ctx, sg.paged(d_a, d_pts[0], job.pools),
                                  sg.paged(d_b, d_pts[1], job.pools),
                                  sg.paged(d_c, d_pts[2], job.pools), 2.5, job.n, job.shift, st)
                sg.colored_gemv(ctx, w, sg.BF16, job.M, job.K_w, d_x, sg.BF16, job.B, d_y, 16, st)
            st.synchronize()
            out[idx] = (d_col.cpu().numpy(), d_hist.cpu().numpy(), d_a.cpu().numpy(),
                        d_y.cpu().numpy())
        sg.stream_release(ctx, st)
    except Exception as e:  # noqa: BLE001 - reported by the test
        out[idx] = e


def test_threads_share_one_context(ctx, orc):
    n_cus = ctx.num_cus
    jobs = [Job(orc, 40 + i) for i in range(4)]
    masks = [range(0, 64), range(64, 128), range(128, 192),
             synth.random_cu_subset(n_cus, 50, seed=3)]
    out = [None] * 4
    say(f"4 host threads, 6 rounds each, masks {[len(list(m)) for m in masks]} CUs")
    threads = [threading.Thread(target=worker, args=(ctx, jobs[i], masks[i], 6, out, i))
               for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
        assert not t.is_alive(), "thread did not finish"
    for i, (job, r) in enumerate(zip(jobs, out)):
        assert not isinstance(r, Exception), (i, r)
        col, hist, a, y = r
        assert (col == job.cols).all(), i
        assert (hist.astype(np.uint64) == job.hist).all(), i
        assert (a.view(np.uint32) == job.a_ref.view(np.uint32)).all(), i
        tp.gemv_check(ctx, y.reshape(job.B, job.M), job.y_ref, job.absdot, job.M, job.K_w, job.B,
                      sg.BF16, sg.BF16, masks[i], tag=f"thread {i}")
    assert ctx.device_error() == 0
