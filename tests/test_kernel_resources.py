"""CPU check of the compiled gfx950 code objects: no library kernel spills
vector registers or uses scratch memory (scalar registers may spill into
vector-register lanes, which stays on chip), and the paged, gated kernels of
the report in tests/resource_report.py compile beside their plain
counterparts."""
import resource_report as rr
from kernel_asm import device_asm, kernel_resources


def test_no_library_kernel_spills():
    for src in ("stream.hip", "gemv.hip", "colour.hip", "context.hip", "bimodal.hip"):
        for name, r in kernel_resources(device_asm(src)).items():
            assert r.get("vgpr_spill", 0) == 0, (name, r)
            assert r.get("scratch", 0) == 0, (name, r)


def test_resource_pairs_compile():
    rows = rr.rows()
    assert len(rows) == len(rr.PAIRS)
    for what, lk, a, pk, b in rows:
        assert a["vgpr"] > 0
        if pk:
            assert b is not None and b["vgpr"] > 0, pk
