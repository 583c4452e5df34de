"""Static check of the built gfx950 code: no workgroup barrier may sit inside
a lane-divergent inner loop of a persistent kernel.

Each kernel's tile loop holds barriers (ticket hand-out, LDS staging).  If a
lane-dependent branch inside the loop body is compiled into an inner loop
that reaches such a barrier (a loop whose back-edge tests the exec mask),
some lanes of a wave can return to the barrier while another lane of the
same wave still owes the next ticket, and the workgroup never finishes.  The
tile bodies are written so that this cannot arise (no early exits, errors
recorded in per-thread bits); an inner loop with a barrier is allowed only
when its trip count is the same for the whole workgroup, which the compiler
shows by closing it with a scalar branch (on SCC or VCC, never on EXEC).
This test compiles every source to gfx950 assembly and checks, for every
barrier at loop depth 2 or more, the back-edges of the inner loops around it.
"""
import re

import pytest

from kernel_asm import device_asm

SOURCES = ["stream.hip", "gemv.hip", "colour.hip", "context.hip"]


def barrier_depths(asm: str):
    """Yield (kernel, depth) for every barrier; depth = loop depth of its block."""
    kernel, depth = None, 0
    for line in asm.splitlines():
        if re.match(r"^_Z\w+:", line):
            kernel, depth = line.split(":")[0], 0
        elif re.match(r"^(\.LBB\d+_\d+:|; %bb\.\d+:)", line):
            depth = 0
            m = re.search(r"Depth=(\d+)", line)
            if m:
                depth = int(m.group(1))
        elif "Depth=" in line and line.lstrip().startswith(";"):
            depth = max(depth, int(re.search(r"Depth=(\d+)", line).group(1)))
        elif re.match(r"^\s+s_barrier\b", line):
            yield kernel, depth


def divergent_barrier_loops(asm: str):
    """Yield (kernel, header) for every inner loop (depth >= 2) that holds a
    barrier and is closed by a branch on the exec mask (or by an indirect
    jump): the loops in which lanes of one wave could part ways."""
    kernel, label, pos = None, None, 0
    headers = {}    # label -> (kernel, position) of inner-loop headers
    branches = []   # (position, opcode, target)
    barriers = []   # (kernel, position)
    for line in asm.splitlines():
        pos += 1
        m = re.match(r"^(_Z\w+):", line)
        if m:
            kernel = m.group(1)
            continue
        m = re.match(r"^(\.LBB\d+_\d+):", line)
        if m:
            label = m.group(1)
        m = re.search(r"Inner Loop Header: Depth=(\d+)", line)
        if m and int(m.group(1)) >= 2 and label is not None:
            headers[label] = (kernel, pos)
        m = re.match(r"^\s+(s_cbranch_\w+|s_branch|s_setpc_b64)\s*(\S*)", line)
        if m:
            branches.append((pos, m.group(1), m.group(2)))
        if re.match(r"^\s+s_barrier\b", line):
            barriers.append((kernel, pos))
    for lab, (k, start) in headers.items():
        back = [(p, op) for p, op, t in branches if t == lab and p > start]
        if not back:
            continue
        end = max(p for p, _ in back)
        if not any(k == bk and start <= bp <= end for bk, bp in barriers):
            continue
        if any(op.startswith("s_cbranch_exec") or op == "s_setpc_b64" for _, op in back):
            yield k, lab


@pytest.mark.parametrize("src", SOURCES)
def test_no_barrier_in_divergent_loop(src):
    asm = device_asm(src)
    found = list(barrier_depths(asm))
    if src != "context.hip":
        assert found, "expected barriers in the persistent kernels"
    bad = sorted(set(divergent_barrier_loops(asm)))
    assert not bad, f"barrier inside a lane-divergent inner loop in: {bad}"


def test_divergent_loop_check_flags_exec_back_edges():
    """The check above on hand-made assembly: a barrier in an inner loop closed
    on EXEC is flagged, one closed on SCC is not, and a barrier outside any
    inner loop is not."""
    def kern(op, barrier_inside=True):
        body = ["_Zk:", ".LBB0_1:  ; =>This Loop Header: Depth=1",
                ".LBB0_2:  ;   Parent Loop BB0_1 Depth=1",
                "          ; =>  This Inner Loop Header: Depth=2",
                "\tv_add_u32 v1, v1, v2"]
        if barrier_inside:
            body.append("\ts_barrier")
        body += [f"\t{op} .LBB0_2", "\ts_barrier" if not barrier_inside else "\ts_nop 0",
                 "\ts_cbranch_scc1 .LBB0_1", "\ts_endpgm"]
        return "\n".join(body)
    assert list(divergent_barrier_loops(kern("s_cbranch_execnz"))) == [("_Zk", ".LBB0_2")]
    assert list(divergent_barrier_loops(kern("s_cbranch_scc0"))) == []
    assert list(divergent_barrier_loops(kern("s_cbranch_vccnz"))) == []
    assert list(divergent_barrier_loops(kern("s_cbranch_execnz", barrier_inside=False))) == []
