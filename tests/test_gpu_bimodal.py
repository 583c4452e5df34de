"""The bimodal tensor runtime on the GPU (paper section 7.2): the forms a
kernel reads and writes by tensor class and co-location state, and the data
moves between page sets, checked byte for byte against the oracle's
relayout and triad."""
import sys

import numpy as np
import pytest

import synth
import paper_2407_13996_amd as sg

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
DEV = "cuda:0"
SHIFT = 16
P = 1 << SHIFT


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
    return torch.from_numpy(a).to(DEV)


def to_host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


class Forms:
    """A tensor of n_pages pages: the all-channel form (identity table over a
    plain buffer) and a coloured form (oracle table of colours S over a
    pool), with host mirrors of both buffers."""

    def __init__(self, orc, n_pages, S, seed, data=None):
        self.n_pages = n_pages
        self.pool_pages = int(n_pages * 64 / len(S) * 1.5) + 16
        masks = synth.xor_masks(6, seed=seed, min_bit=SHIFT)
        self.pt_part, found = orc.pagetable(masks, 0, SHIFT, self.pool_pages,
                                            synth.colour_set_bits(S), n_pages)
        assert found >= n_pages
        self.pt_all = np.arange(n_pages, dtype=np.uint32)
        self.h_all = data if data is not None else np.zeros(n_pages * P // 4, np.float32)
        self.d_all = to_dev(self.h_all)
        self.d_part = torch.zeros(self.pool_pages * P // 4, dtype=torch.float32, device=DEV)
        self.d_pt_all, self.d_pt_part = to_dev(self.pt_all), to_dev(self.pt_part)
        self.all = sg.paged(self.d_all, self.d_pt_all, n_pages)
        self.part = sg.paged(self.d_part, self.d_pt_part, self.pool_pages)

    def part_as_logical(self):
        """The part form's contents gathered back to logical order."""
        pool = to_host(self.d_part).reshape(self.pool_pages, P // 4)
        return pool[self.pt_part.astype(np.int64)].reshape(-1)


def same_bits(a, b):
    return (np.asarray(a).view(np.uint32) == np.asarray(b).view(np.uint32)).all()


def triad(ctx, a, b, c, n, stream=None):
    sg.colored_stream(ctx, a, b, c, 3.0, n, SHIFT, stream)


def test_be_weight_two_copies_and_state_selection(ctx, orc):
    n_pages = 24
    n = n_pages * P // 4
    w = Forms(orc, n_pages, range(48, 64), seed=1, data=synth.uniform_f32(n, seed=2))
    c = Forms(orc, n_pages, range(48, 64), seed=1, data=synth.uniform_f32(n, seed=3))
    out = Forms(orc, n_pages, range(48, 64), seed=1)
    bm = sg.Bimodal(ctx)
    try:
        wid = bm.register(sg.BM_BE_WEIGHT, w.all, w.part, n * 4, SHIFT)
        cid = bm.register(sg.BM_BE_WEIGHT, c.all, c.part, n * 4, SHIFT)
        assert same_bits(w.part_as_logical(), w.h_all)          # the second resident copy
        ref = w.h_all.copy()
        orc.triad(ref, np.arange(n_pages, dtype=np.uint32), w.h_all, w.pt_all, c.h_all, c.pt_all,
                  3.0, n, SHIFT)
        for state, form in ((sg.BM_MONOPOLY, sg.BM_ALL), (sg.BM_COLOCATED, sg.BM_PART)):
            bm.set_state(state)
            (bw, fw), (bc, fc) = bm.input(wid), bm.input(cid)
            assert fw == fc == form
            out.d_all.zero_()
            triad(ctx, out.all, bw, bc, n)
            assert same_bits(to_host(out.d_all), ref), state
        with pytest.raises(sg.SgdrcError):
            bm.output(wid)                                      # weights are read-only
    finally:
        bm.close()


def test_ls_tensor_moves_with_the_state(ctx, orc):
    n_pages = 40
    n = n_pages * P // 4
    data = synth.uniform_f32(n, seed=7)
    x = Forms(orc, n_pages, range(0, 48), seed=4, data=data)
    bm = sg.Bimodal(ctx)
    try:
        tid = bm.register(sg.BM_LS_TENSOR, x.all, x.part, n * 4, SHIFT)
        assert bm.input(tid)[1] == sg.BM_ALL
        bm.set_state(sg.BM_COLOCATED)
        assert bm.input(tid)[1] == sg.BM_PART and bm.output(tid)[1] == sg.BM_PART
        assert same_bits(x.part_as_logical(), data)
        x.d_all.zero_()                                         # the old form is free now
        bm.set_state(sg.BM_MONOPOLY)
        assert bm.input(tid)[1] == sg.BM_ALL
        assert same_bits(to_host(x.d_all), data)
        # registered while colocated: moved at once
        y = Forms(orc, n_pages, range(0, 48), seed=5, data=synth.uniform_f32(n, seed=8))
        bm.set_state(sg.BM_COLOCATED)
        yid = bm.register(sg.BM_LS_TENSOR, y.all, y.part, n * 4, SHIFT)
        assert bm.input(yid)[1] == sg.BM_PART
        assert same_bits(y.part_as_logical(), y.h_all)
        assert same_bits(x.part_as_logical(), data)            # x moved again with the state
    finally:
        bm.close()


def test_activation_read_where_its_writer_left_it(ctx, orc):
    """Two chained BE triads: the first writes activation A while colocated
    (BE channels); the state turns to monopolization; the second reads A
    from the BE channels (its writer's form) and writes B over all channels."""
    n_pages = 32
    n = n_pages * P // 4 - 5                                    # ragged tail
    b = Forms(orc, n_pages, range(48, 64), seed=9, data=synth.uniform_f32(n_pages * P // 4, seed=10))
    c = Forms(orc, n_pages, range(48, 64), seed=9, data=synth.uniform_f32(n_pages * P // 4, seed=11))
    A = Forms(orc, n_pages, range(48, 64), seed=9)
    B = Forms(orc, n_pages, range(48, 64), seed=9)
    bm = sg.Bimodal(ctx)
    try:
        wb = bm.register(sg.BM_BE_WEIGHT, b.all, b.part, n_pages * P, SHIFT)
        wc = bm.register(sg.BM_BE_WEIGHT, c.all, c.part, n_pages * P, SHIFT)
        ia = bm.register(sg.BM_ACTIVATION, A.all, A.part, n_pages * P, SHIFT)
        ib = bm.register(sg.BM_ACTIVATION, B.all, B.part, n_pages * P, SHIFT)
        a_id, b_id = bm.acquire(n * 4), bm.acquire(n * 4)
        assert {a_id, b_id} == {ia, ib}
        bm.set_state(sg.BM_COLOCATED)
        oa, fa = bm.output(a_id)
        assert fa == sg.BM_PART
        triad(ctx, oa, bm.input(wb)[0], bm.input(wc)[0], n)
        bm.set_state(sg.BM_MONOPOLY)
        ra, fra = bm.input(a_id)
        assert fra == sg.BM_PART                                # where it was written
        ob, fb = bm.output(b_id)
        assert fb == sg.BM_ALL
        triad(ctx, ob, ra, bm.input(wc)[0], n)
        # oracle: A = b + 3c, B = A + 3c (logical order, identity tables)
        ident = np.arange(n_pages, dtype=np.uint32)
        ref_a = np.zeros(n_pages * P // 4, np.float32)
        orc.triad(ref_a, ident, b.h_all, ident, c.h_all, ident, 3.0, n, SHIFT)
        ref_b = np.zeros(n_pages * P // 4, np.float32)
        orc.triad(ref_b, ident, ref_a, ident, c.h_all, ident, 3.0, n, SHIFT)
        got_a = (A.part_as_logical() if a_id == ia else B.part_as_logical())
        got_b = to_host((B if b_id == ib else A).d_all)
        assert same_bits(got_a[:n], ref_a[:n])
        assert same_bits(got_b[:n], ref_b[:n])
        bm.release(a_id)
        assert bm.acquire(1) == a_id                            # A's buffer reused
    finally:
        bm.close()
