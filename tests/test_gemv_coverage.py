"""CPU check: every GEMV kernel variant a benchmark configuration launches
is launched by some GPU parity test as well.  The variant comes from the
library's host-only plan query (colored_gemv_plan), the same function
colored_gemv launches by."""
import pytest

import gemv_cases as gc

sg = pytest.importorskip("paper_2407_13996_amd")


def _variant(case):
    M, K, B, wd, xd, shift, cus = case
    p = sg.gemv_plan(gc.NUM_CUS if cus is None else cus, wd, M, K, xd, B)
    esize = 4 if wd == gc.F32 else 2
    whole = -(-(M * K * esize) // (1 << shift)) <= 256   # table staged once per workgroup
    return (p["path"], p["rows"], p["loads"], p["batch_cols"], p["x_once"], wd, xd, whole)


def test_every_benchmarked_gemv_variant_is_gpu_tested():
    tested = {_variant(c) for c in gc.gpu_cases()}
    missing = {}
    for c in gc.bench_cases():
        v = _variant(c)
        if v not in tested:
            missing[v] = c
    assert not missing, f"benchmarked GEMV variants no GPU test reaches: {missing}"


def test_plan_matches_the_c3_sweep_expectations():
    """The two LS layers (4096x11008, 11008x4096) at batch 1 and 8 on 256 CUs: the vector path with
    two-row tiles for 4096 x 11008 batch 1 (six loads per lane: one round
    over a 22 KB row), MFMA from batch 3 on, and a summation depth far below
    the 1e-3 criterion's K."""
    p = sg.gemv_plan(256, gc.BF16, 4096, 11008, gc.BF16, 1)
    assert (p["path"], p["rows"], p["loads"]) == ("valu", 2, 6)
    assert p["tiles"] == 2048
    q = sg.gemv_plan(256, gc.BF16, 11008, 4096, gc.BF16, 8)
    assert q["path"] == "mfma" and q["tiles"] == 11008 // q["rows"]
    for r in (p, q):
        assert 0 < r["sum_depth"] < 200


def test_plan_rejects_bad_arguments():
    with pytest.raises(sg.SgdrcError):
        sg.gemv_plan(0, gc.BF16, 16, 16, gc.BF16, 1)
    with pytest.raises(sg.SgdrcError):
        sg.gemv_plan(257, gc.BF16, 16, 16, gc.BF16, 1)
    with pytest.raises(sg.SgdrcError):
        sg.gemv_plan(64, gc.BF16, 16, 12, gc.BF16, 1)     # K * 2 not a multiple of 16
    with pytest.raises(sg.SgdrcError):
        sg.gemv_plan(64, gc.BF16, 16, 16, gc.BF16, 9)


def test_plan_x_once_rules():
    """Which launches load x once per workgroup: vector path when one round
    of loads covers a row and x is half a tile's bytes (W and x of one
    type); MFMA path at batch 3-4 with rows of at most 8 KiB."""
    for cus in (64, 128, 192, 256):
        p = sg.gemv_plan(cus, gc.BF16, 4096, 11008, gc.BF16, 1)
        assert (p["path"], p["rows"], p["loads"], p["x_once"]) == ("valu", 2, 6, True), (cus, p)
        assert not sg.gemv_plan(cus, gc.BF16, 4096, 11008, gc.F32, 1)["x_once"]
        assert not sg.gemv_plan(cus, gc.BF16, 11008, 4096, gc.BF16, 1)["x_once"]   # x a quarter
        assert sg.gemv_plan(cus, gc.BF16, 11008, 4096, gc.BF16, 2)["x_once"]
        assert not sg.gemv_plan(cus, gc.BF16, 4096, 11008, gc.BF16, 2)["x_once"]   # two rounds
        q = sg.gemv_plan(cus, gc.BF16, 11008, 4096, gc.BF16, 4)
        assert q["path"] == "mfma" and q["batch_cols"] == 4 and q["x_once"], (cus, q)
        assert not sg.gemv_plan(cus, gc.BF16, 4096, 11008, gc.BF16, 4)["x_once"]   # 22 KB rows
        assert not sg.gemv_plan(cus, gc.BF16, 11008, 4096, gc.BF16, 8)["x_once"]   # eight x rows
    # rows longer than six loads per lane cover keep per-tile x
    assert not sg.gemv_plan(256, gc.BF16, 512, 16384, gc.BF16, 1)["x_once"]
