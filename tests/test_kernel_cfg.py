"""Static check of the built gfx950 code: no workgroup barrier may sit inside
a nested loop of a persistent kernel.

Each kernel's tile loop holds barriers (ticket hand-out, LDS staging).  If a
lane-dependent branch inside the loop body is compiled into an inner loop
that reaches such a barrier, some lanes of a wave can return to the barrier
while another lane of the same wave still owes the next ticket, and the
workgroup never finishes.  The tile bodies are written so that this cannot
arise (no early exits, errors recorded in per-thread bits); this test
compiles every source to gfx950 assembly and checks the loop depth that the
compiler reports for every block containing a barrier.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_13996_amd", "csrc")
SOURCES = ["stream.hip", "gemv.hip", "colour.hip", "context.hip"]


def device_asm(src: str, tmp_path) -> str:
    out = tmp_path / (os.path.splitext(src)[0] + ".s")
    cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "--cuda-device-only", "-S", "-O3",
           "-std=c++17", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, src), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return out.read_text()


def barrier_depths(asm: str):
    """Yield (kernel, depth) for every barrier; depth = loop depth of its block."""
    kernel, depth = None, 0
    for line in asm.splitlines():
        if re.match(r"^_Z\w+:", line):
            kernel, depth = line[:-1], 0
        elif re.match(r"^(\.LBB\d+_\d+:|; %bb\.\d+:)", line):
            depth = 0
            m = re.search(r"Depth=(\d+)", line)
            if m:
                depth = int(m.group(1))
        elif "Depth=" in line and line.lstrip().startswith(";"):
            depth = max(depth, int(re.search(r"Depth=(\d+)", line).group(1)))
        elif re.match(r"^\s+s_barrier\b", line):
            yield kernel, depth


@pytest.mark.parametrize("src", SOURCES)
def test_no_barrier_in_nested_loop(src, tmp_path):
    asm = device_asm(src, tmp_path)
    found = list(barrier_depths(asm))
    if src != "context.hip":
        assert found, "expected barriers in the persistent kernels"
    bad = sorted(set(k for k, d in found if d >= 2))
    assert not bad, f"barrier inside a nested loop in: {bad}"
