"""Registers and LDS of the library's paged, CU-gated kernels beside plain
contiguous counterparts (tests/plain_kernels.hip) with the same per-lane
work: what page indirection and the gate cost in resources, the analogue of
the count of extra registers that re-indexing adds (paper section 9.1.2).

    python tests/resource_report.py        # prints a markdown table
"""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

from kernel_asm import PLAIN, device_asm, kernel_resources  # noqa: E402

# (what, library kernel, source, plain kernel)
PAIRS = [
    ("triad, 16 slices per lane and array", "sgdrc::k_triad<16, false>", "stream.hip", "plain_triad<16>"),
    ("triad, preemptible", "sgdrc::k_triad<16, true>", "stream.hip", "plain_triad<16>"),
    ("relayout (copy), 16 slices per lane", "sgdrc::k_relayout<16, false>", "stream.hip", "plain_copy<16>"),
    ("GEMV batch 1, 2 rows x 6 slices", "sgdrc::k_gemv_valu<1, 1, 1, 2, 6, false>", "gemv.hip", "plain_gemv<2, 6>"),
    ("GEMV batch 1, 2 rows x 6 slices, x once per workgroup", "sgdrc::k_gemv_valu<1, 1, 1, 2, 6, true>", "gemv.hip",
     "plain_gemv<2, 6>"),
    ("GEMV batch 1, 4 rows x 3 slices", "sgdrc::k_gemv_valu<1, 1, 1, 4, 3, false>", "gemv.hip", "plain_gemv<4, 3>"),
    ("GEMV batch 1, 4 rows x 2 slices", "sgdrc::k_gemv_valu<1, 1, 1, 4, 2, false>", "gemv.hip", "plain_gemv<4, 2>"),
    ("GEMV batch 5-8, MFMA 16-row tiles", "sgdrc::k_gemm_mfma<1, 16, 8, false>", "gemv.hip", None),
    ("GEMV batch 3-4, MFMA 16-row tiles", "sgdrc::k_gemm_mfma<1, 16, 4, false>", "gemv.hip", None),
    ("GEMV batch 3-4, MFMA 16-row tiles, x for the whole K in LDS", "sgdrc::k_gemm_mfma<1, 16, 4, true>", "gemv.hip",
     None),
    ("classify, 8 loads per lane", "sgdrc::k_classify<6, false, false>", "colour.hip", "plain_classify<8>"),
    ("classify + histogram", "sgdrc::k_classify<6, true, false>", "colour.hip", "plain_classify<8>"),
]


def waves_per_simd(vgpr: int, agpr: int) -> int:
    """Waves a SIMD holds by register file (512 registers per lane, allocated in
    blocks of 8)."""
    regs = -(-(vgpr + agpr) // 8) * 8
    return max(0, min(8, 512 // max(regs, 1)))


def rows():
    lib = {}
    for src in sorted({p[2] for p in PAIRS}):
        lib.update(kernel_resources(device_asm(src)))
    plain = kernel_resources(device_asm(PLAIN))
    out = []
    for what, lk, src, pk in PAIRS:
        a = lib[lk]
        b = plain.get(pk) if pk else None
        out.append((what, lk, a, pk, b))
    return out


def main():
    print("| kernel | library VGPR / SGPR / LDS B / spills | plain VGPR / SGPR / LDS B | extra VGPR | "
          "waves per SIMD (library / plain) |")
    print("|---|---|---|---:|---|")
    for what, lk, a, pk, b in rows():
        la = f"{a['vgpr'] + a.get('agpr', 0)} / {a['sgpr']} / {a['lds']} / {a.get('vgpr_spill', 0) + a.get('sgpr_spill', 0)}"
        if b:
            pa = f"{b['vgpr'] + b.get('agpr', 0)} / {b['sgpr']} / {b['lds']}"
            extra = f"{a['vgpr'] + a.get('agpr', 0) - b['vgpr'] - b.get('agpr', 0):+d}"
            wv = f"{waves_per_simd(a['vgpr'], a.get('agpr', 0))} / {waves_per_simd(b['vgpr'], b.get('agpr', 0))}"
        else:
            pa, extra, wv = "—", "—", f"{waves_per_simd(a['vgpr'], a.get('agpr', 0))} / —"
        print(f"| {what}: `{lk}` vs `{pk or '—'}` | {la} | {pa} | {extra} | {wv} |")


if __name__ == "__main__":
    main()
