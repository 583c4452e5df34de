"""C-ABI checks that need no GPU: the library loads, exports every function
declared in include/sgdrc.h, and rejects bad arguments on the host before
touching the device (arguments are checked before the context, so a NULL
context still reports EINVAL for a bad argument and ENODEV otherwise)."""
import ctypes
import os
import re

import pytest

import paper_2407_13996_amd as sg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sgdrc.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while")))


@pytest.fixture(scope="module")
def L():
    return sg.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ["colour_classify", "colour_alloc_pagetable", "bimodal_relayout", "colored_stream",
              "colored_gemv", "set_cu_mask", "sgdrc_init", "sgdrc_destroy"]:
        assert n in names


def test_library_exports_every_declared_symbol(L):
    missing = [n for n in declared_functions() if not hasattr(L, n)]
    assert not missing, missing


def test_library_exports_nothing_else():
    """The dynamic symbol table's functions are exactly the header's (the
    link's version script keeps the C++ internals local)."""
    import shutil
    import subprocess
    nm = shutil.which("nm") or shutil.which("llvm-nm") or "/opt/rocm/llvm/bin/llvm-nm"
    out = subprocess.run([nm, "-D", "--defined-only", sg.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(line.split()[-1] for line in out.splitlines() if " T " in line)
    assert exported == declared_functions()


NULL = None


def good_hash(k=4):
    return sg.make_hash([1 << (16 + i) for i in range(k)])


def test_classify_argument_errors(L):
    h = good_hash()
    assert L.colour_classify(NULL, None, 16, 1, 32, None, None) == sg.EINVAL   # NULL hash
    bad = good_hash(); bad.n_masks = 0
    assert L.colour_classify(NULL, ctypes.byref(bad), 16, 1, 32, None, None) == sg.EINVAL
    bad = good_hash(); bad.n_masks = 9
    assert L.colour_classify(NULL, ctypes.byref(bad), 16, 1, 32, None, None) == sg.EINVAL
    bad = good_hash(); bad.masks[0] = 1 << 48
    assert L.colour_classify(NULL, ctypes.byref(bad), 16, 1, 32, None, None) == sg.EINVAL
    assert "47" in sg.last_error()
    assert L.colour_classify(NULL, ctypes.byref(h), 8, 1, 32, None, None) == sg.EINVAL  # misaligned
    assert L.colour_classify(NULL, ctypes.byref(h), 0, 5, 32, None, None) == sg.EINVAL  # NULL addrs
    assert L.colour_classify(NULL, ctypes.byref(h), 16, 1, 32, None, None) == sg.ENODEV
    assert L.colour_classify(NULL, ctypes.byref(h), 0, 0, 0, None, None) == sg.ENODEV   # n = 0 ok


def call_pt(L, h, origin=0, shift=16, pool=1024, colours=(0,), n=8, pt=256, found=True):
    f = ctypes.c_uint64()
    s = sg.make_set(sg.words_of(colours))
    return L.colour_alloc_pagetable(NULL, ctypes.byref(h) if h is not None else None, origin, shift,
                                    pool, ctypes.byref(s), n, pt,
                                    ctypes.byref(f) if found else None, None)


def test_pagetable_argument_errors(L):
    h = good_hash(4)
    assert call_pt(L, h) == sg.ENODEV
    assert call_pt(L, None) == sg.EINVAL
    assert call_pt(L, h, shift=9) == sg.EINVAL
    assert call_pt(L, h, shift=31) == sg.EINVAL
    assert call_pt(L, h, origin=4096, shift=16) == sg.EINVAL          # origin not page aligned
    assert call_pt(L, h, colours=(16,)) == sg.EINVAL                  # colour >= 2^K
    assert call_pt(L, h, colours=()) == sg.EINVAL                     # empty set
    assert call_pt(L, h, n=2000) == sg.EINVAL                         # n_needed > pool_pages
    assert call_pt(L, h, pool=0) == sg.EINVAL
    assert call_pt(L, h, pool=(1 << 32) + 1) == sg.EINVAL
    assert call_pt(L, h, origin=(1 << 48) - (1 << 16), pool=2) == sg.EINVAL  # past 2^48
    assert call_pt(L, h, pt=None) == sg.EINVAL
    assert call_pt(L, h, found=False) == sg.EINVAL


def pg(pool=256, pt=256, pages=4):
    return sg.Paged(pool, pt, pages)


def test_relayout_and_stream_argument_errors(L):
    r = ctypes.byref
    assert L.bimodal_relayout(NULL, r(pg()), r(pg()), 100, 16, None) == sg.ENODEV
    assert L.bimodal_relayout(NULL, r(pg()), r(pg()), 100, 9, None) == sg.EINVAL
    assert L.bimodal_relayout(NULL, r(pg(pool=128)), r(pg()), 100, 16, None) == sg.EINVAL
    assert L.bimodal_relayout(NULL, r(pg(pt=0)), r(pg()), 100, 16, None) == sg.EINVAL
    assert L.bimodal_relayout(NULL, r(pg(pages=0)), r(pg()), 100, 16, None) == sg.EINVAL
    assert L.bimodal_relayout(NULL, None, r(pg()), 100, 16, None) == sg.EINVAL
    assert L.colored_stream(NULL, r(pg()), r(pg()), r(pg()), 3.0, 100, 16, None) == sg.ENODEV
    assert L.colored_stream(NULL, r(pg()), r(pg(pt=2)), r(pg()), 3.0, 100, 16, None) == sg.EINVAL


def test_relayout_batch_argument_errors(L):
    def items(*its):
        arr = (sg.RelayoutItem * max(len(its), 1))()
        for i, it in enumerate(its):
            arr[i] = it
        return arr, len(its)

    ok = sg.RelayoutItem(pg(), pg(), 100, 16, 0)
    a, n = items(ok, ok)
    assert L.bimodal_relayout_batch(NULL, a, n, None) == sg.ENODEV
    assert L.bimodal_relayout_batch(NULL, None, 0, None) == sg.ENODEV      # nothing to check
    assert L.bimodal_relayout_batch(NULL, None, 3, None) == sg.EINVAL
    for bad in (sg.RelayoutItem(pg(), pg(), 100, 9, 0), sg.RelayoutItem(pg(), pg(), 100, 31, 0),
                sg.RelayoutItem(pg(pool=128), pg(), 100, 16, 0),
                sg.RelayoutItem(pg(), pg(pt=0), 100, 16, 0),
                sg.RelayoutItem(pg(), pg(pages=0), 100, 16, 0),
                sg.RelayoutItem(pg(), pg(), 100, 16, 1),                   # reserved
                sg.RelayoutItem(pg(), pg(), 1 << 62, 16, 0)):             # too many tiles
        a, n = items(ok, bad)
        assert L.bimodal_relayout_batch(NULL, a, n, None) == sg.EINVAL
        assert "item 1" in L.sgdrc_last_error().decode()


def test_gemv_argument_errors(L):
    r = ctypes.byref
    w = pg()
    ok = dict(wd=sg.BF16, M=64, K=64, xd=sg.BF16, b=1, x=256, y=256, shift=21)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return L.colored_gemv(NULL, r(w), a["wd"], a["M"], a["K"], a["x"], a["xd"], a["b"], a["y"],
                              a["shift"], None)
    assert call() == sg.ENODEV
    assert call(b=0) == sg.EINVAL
    assert call(b=9) == sg.EINVAL
    assert call(wd=3) == sg.EINVAL
    assert call(xd=-1) == sg.EINVAL
    assert call(M=0) == sg.EINVAL
    assert call(K=12) == sg.EINVAL          # 24 bytes per row: not a multiple of 16
    assert call(wd=sg.F32, K=12) == sg.ENODEV
    assert call(x=0) == sg.EINVAL
    assert call(x=264) == sg.EINVAL         # x not 16-byte aligned
    assert call(shift=40) == sg.EINVAL
    assert call(K=1 << 28, b=8) == sg.EINVAL  # x of 4 GiB
    assert call(K=1 << 28, b=7) == sg.EINVAL  # a 16-row tile spans 4096 pages of 2 MiB
    assert call(K=1 << 20, b=7) == sg.ENODEV  # 16 pages per tile: fine


def test_context_calls_reject_null(L):
    assert L.sgdrc_num_cus(NULL) == sg.ENODEV
    m = sg.make_set([0, 0, 0, 0], sg.CuMask)
    assert L.set_cu_mask(NULL, None, ctypes.byref(m)) == sg.EINVAL     # empty mask
    m = sg.make_set([1, 0, 0, 0], sg.CuMask)
    assert L.set_cu_mask(NULL, None, ctypes.byref(m)) == sg.ENODEV
    f = ctypes.c_uint32()
    assert L.sgdrc_device_error(NULL, ctypes.byref(f)) == sg.ENODEV
    assert L.sgdrc_init(0, None) == sg.EINVAL
    assert L.sgdrc_set_timelog(NULL, None, 256, 0) == sg.EINVAL        # slots but n_slots 0
    assert L.sgdrc_set_timelog(NULL, None, 260, 4) == sg.EINVAL        # misaligned slots
    assert L.sgdrc_set_timelog(NULL, None, 256, 4) == sg.ENODEV
    assert L.sgdrc_set_timelog(NULL, None, None, 0) == sg.ENODEV       # off, but no context
    k = ctypes.c_uint32()
    assert L.sgdrc_wallclock_khz(NULL, None) == sg.EINVAL
    assert L.sgdrc_wallclock_khz(NULL, ctypes.byref(k)) == sg.ENODEV


def test_binding_raises_with_message():
    with pytest.raises(sg.SgdrcError) as e:
        sg.set_cu_mask(None, 0, [])
    assert e.value.code == sg.EINVAL and "empty" in str(e.value)


def test_preemption_argument_errors(L):
    t = ctypes.c_uint64()
    assert L.sgdrc_set_eviction_flag(NULL, None, 258) == sg.EINVAL     # misaligned flag
    assert L.sgdrc_set_eviction_flag(NULL, None, 256) == sg.ENODEV
    assert L.sgdrc_set_eviction_flag(NULL, None, None) == sg.ENODEV
    assert L.sgdrc_resume(NULL, None) == sg.ENODEV
    assert L.sgdrc_suspended(NULL, None, None) == sg.EINVAL
    assert L.sgdrc_suspended(NULL, None, ctypes.byref(t)) == sg.ENODEV
    assert L.sgdrc_signal_flag(NULL, None, None, 1, None) == sg.EINVAL    # NULL flag
    assert L.sgdrc_signal_flag(NULL, None, 258, 1, None) == sg.EINVAL     # misaligned flag
    assert L.sgdrc_signal_flag(NULL, None, 256, 1, 260) == sg.EINVAL      # misaligned stamp
    assert L.sgdrc_signal_flag(NULL, None, 256, 1, 264) == sg.ENODEV


# ------------------------------------------------- sliding-window reservation
# The CUs reserved for latency-sensitive kernels are the most that any
# kernel in the window of the next queued ones needs (paper section 7.1),
# here rounded up to a granule and given as the first logical CUs.

def test_tidal_masks_hand_worked():
    # queue needs 24, 64, 8 CUs: a window of 1 sees 24, of 2 or more 64
    assert sg.tidal_masks(256, [24, 64, 8], window=1)[0] == list(range(24))
    assert sg.tidal_masks(256, [24, 64, 8], window=2)[0] == list(range(64))
    assert sg.tidal_masks(256, [24, 64, 8], window=9)[0] == list(range(64))
    # whole XCDs: 24 -> 32, 65 -> 96
    assert sg.tidal_masks(256, [24], window=1, granule=32)[0] == list(range(32))
    assert sg.tidal_masks(256, [65, 3], window=2, granule=32)[0] == list(range(96))
    # nothing queued: everything to the best-effort side
    ls, be = sg.tidal_masks(256, [], window=4)
    assert ls == [] and be == list(range(256))
    # a need of the whole device leaves the best-effort side empty
    ls, be = sg.tidal_masks(256, [10, 256], window=2)
    assert ls == list(range(256)) and be == []
    # rounding never exceeds the device
    assert sg.tidal_masks(250, [249], window=1, granule=32)[0] == list(range(250))


def test_tidal_masks_partition_random_queues():
    import numpy as np
    rng = np.random.default_rng(11)
    for _ in range(200):
        n = int(rng.integers(1, 257))
        q = [int(x) for x in rng.integers(0, n + 1, size=int(rng.integers(0, 12)))]
        w = int(rng.integers(1, 6))
        gr = int(rng.choice([1, 8, 32]))
        ls, be = sg.tidal_masks(n, q, window=w, granule=gr)
        assert sorted(ls + be) == list(range(n))           # a partition of the CUs
        assert ls == list(range(len(ls)))                   # LS holds a prefix
        r = len(ls)
        need = max(q[:w], default=0)
        assert r >= need and (r == n or r % gr == 0) and r - need < gr


def test_tidal_masks_argument_errors(L):
    ls, be = sg.CuMask(), sg.CuMask()
    r = ctypes.byref
    q = (ctypes.c_uint32 * 2)(4, 8)
    assert L.sgdrc_tidal_masks(0, q, 2, 1, 1, r(ls), r(be)) == sg.EINVAL
    assert L.sgdrc_tidal_masks(257, q, 2, 1, 1, r(ls), r(be)) == sg.EINVAL
    assert L.sgdrc_tidal_masks(256, q, 2, 0, 1, r(ls), r(be)) == sg.EINVAL
    assert L.sgdrc_tidal_masks(256, q, 2, 1, 0, r(ls), r(be)) == sg.EINVAL
    assert L.sgdrc_tidal_masks(256, None, 2, 1, 1, r(ls), r(be)) == sg.EINVAL
    assert L.sgdrc_tidal_masks(4, q, 2, 2, 1, r(ls), r(be)) == sg.EINVAL   # 8 > 4 CUs
    assert L.sgdrc_tidal_masks(256, q, 2, 1, 1, None, r(be)) == sg.EINVAL
    assert L.sgdrc_tidal_masks(256, q, 2, 1, 1, r(ls), r(be)) == sg.OK


# ------------------------------------------------------ bimodal runtime (host)
# A runtime without context holds activations only, which is enough to check
# the section 7.2 rules that need no data movement: an intermediate result is
# written in the form of the writing kernel's state and read from where it
# was last written, and buffers are reused smallest-fit.

def _forms(base):
    return sg.Paged(base, base + 4096, 8), sg.Paged(base + (1 << 20), base + (1 << 20) + 4096, 8)


def test_bimodal_activation_follows_its_writer():
    bm = sg.Bimodal(None)
    try:
        a, p = _forms(1 << 32)
        t = bm.register(sg.BM_ACTIVATION, a, p, 4096, 12)
        with pytest.raises(sg.SgdrcError):
            bm.input(t)                                    # never written
        assert bm.state == sg.BM_MONOPOLY
        desc, w = bm.output(t)
        assert w == sg.BM_ALL and desc.pool == a.pool and desc.pt == a.pt
        bm.set_state(sg.BM_COLOCATED)
        assert bm.input(t)[1] == sg.BM_ALL                 # read where written
        desc, w = bm.output(t)
        assert w == sg.BM_PART and desc.pool == p.pool
        bm.set_state(sg.BM_MONOPOLY)
        assert bm.input(t)[1] == sg.BM_PART
        bm.set_state(sg.BM_MONOPOLY)                       # no change, no effect
        assert bm.state == sg.BM_MONOPOLY
    finally:
        bm.close()


def test_bimodal_activation_reuse_smallest_fit():
    bm = sg.Bimodal(None)
    try:
        ids = [bm.register(sg.BM_ACTIVATION, *_forms(1 << 32), cap, 12)
               for cap in (1 << 20, 4 << 20, 2 << 20, 2 << 20)]
        assert ids == [0, 1, 2, 3]
        assert bm.acquire(3 << 19) == 2                    # 1.5 MiB -> first 2 MiB buffer
        assert bm.acquire(3 << 19) == 3
        assert bm.acquire(3 << 19) == 1                    # then the 4 MiB one
        with pytest.raises(sg.SgdrcError) as e:
            bm.acquire(3 << 19)
        assert e.value.code == sg.ENOMEM
        assert bm.acquire(1) == 0
        bm.output(2)
        bm.release(2)
        assert bm.acquire(100) == 2                        # reused, contents unwritten
        with pytest.raises(sg.SgdrcError):
            bm.input(2)
        with pytest.raises(sg.SgdrcError):
            bm.release(0) or bm.release(0)                 # second release of 0 fails
    finally:
        bm.close()


def test_bimodal_argument_errors(L):
    r = ctypes.byref
    h = ctypes.c_void_p()
    assert L.sgdrc_bm_create(NULL, None) == sg.EINVAL
    assert L.sgdrc_bm_create(NULL, r(h)) == sg.OK
    i = ctypes.c_uint32()
    a, p = _forms(1 << 32)
    assert L.sgdrc_bm_register(h, 3, r(a), r(p), 64, 12, None, r(i)) == sg.EINVAL      # class
    assert L.sgdrc_bm_register(h, 2, r(a), r(p), 0, 12, None, r(i)) == sg.EINVAL       # 0 bytes
    assert L.sgdrc_bm_register(h, 2, r(a), r(p), 64, 9, None, r(i)) == sg.EINVAL       # shift
    assert L.sgdrc_bm_register(h, 2, None, r(p), 64, 12, None, r(i)) == sg.EINVAL
    assert L.sgdrc_bm_register(h, 0, r(a), r(p), 64, 12, None, r(i)) == sg.ENODEV      # no ctx
    assert L.sgdrc_bm_register(h, 1, r(a), r(p), 64, 12, None, r(i)) == sg.ENODEV
    assert L.sgdrc_bm_set_state(h, 2, None) == sg.EINVAL
    out = sg.Paged()
    assert L.sgdrc_bm_input(h, 0, r(out), None) == sg.EINVAL                           # no id 0
    assert L.sgdrc_bm_register(h, 2, r(a), r(p), 64, 12, None, r(i)) == sg.OK
    assert L.sgdrc_bm_output(h, 0, None, None) == sg.EINVAL
    assert L.sgdrc_bm_release(h, 0) == sg.EINVAL                                       # not acquired
    assert L.sgdrc_bm_destroy(h) == sg.OK
    assert L.sgdrc_bm_input(None, 0, r(out), None) == sg.EINVAL


def test_colour_table_argument_errors(L):
    r = ctypes.byref
    t = sg.ColourTable(4096, 0, 100, 10, 0)
    s = sg.make_set(sg.words_of([1, 2]))
    f = ctypes.c_uint64()
    assert L.colour_classify_table(NULL, r(t), 16, 1, 32, None, None) == sg.ENODEV
    assert L.colour_classify_table(NULL, None, 16, 1, 32, None, None) == sg.EINVAL
    for bad in (sg.ColourTable(4096, 0, 100, 7, 0), sg.ColourTable(4096, 0, 100, 31, 0),
                sg.ColourTable(4096, 0, 100, 10, 1), sg.ColourTable(None, 0, 100, 10, 0),
                sg.ColourTable(4096, (1 << 48) - 1024, 2, 10, 0)):
        assert L.colour_classify_table(NULL, r(bad), 16, 1, 32, None, None) == sg.EINVAL
    assert L.colour_classify_table(NULL, r(sg.ColourTable(None, 0, 0, 10, 0)), 16, 1, 32, None,
                                   None) == sg.ENODEV                       # empty table is fine
    assert L.colour_classify_table(NULL, r(t), 8, 1, 32, None, None) == sg.EINVAL   # misaligned
    assert L.colour_alloc_pagetable_table(NULL, r(t), 0, 12, 64, r(s), 8, 256, r(f), None) == sg.ENODEV
    assert L.colour_alloc_pagetable_table(NULL, r(t), 0, 9, 64, r(s), 8, 256, r(f), None) == sg.EINVAL
    s255 = sg.make_set(sg.words_of([255]))
    assert L.colour_alloc_pagetable_table(NULL, r(t), 0, 12, 64, r(s255), 8, 256, r(f), None) == sg.EINVAL
    assert L.colour_alloc_pagetable_table(NULL, r(t), 100, 12, 64, r(s), 8, 256, r(f), None) == sg.EINVAL
    assert L.colour_alloc_pagetable_table(NULL, r(t), 0, 12, 64, r(s), 80, 256, r(f), None) == sg.EINVAL
