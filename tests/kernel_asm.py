"""gfx950 assembly of the library's sources (and of tests/plain_kernels.hip),
compiled once per process with the library's own flags, and the per-kernel
resource records of its code-object metadata."""
import os
import re
import subprocess
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_13996_amd", "csrc")
PLAIN = os.path.join(ROOT, "tests", "plain_kernels.hip")
_CACHE = {}
_DIR = None


def device_asm(path: str) -> str:
    """gfx950 assembly of a HIP source (a name in csrc/ or a path)."""
    global _DIR
    if not os.path.isabs(path):
        path = os.path.join(CSRC, path)
    if path not in _CACHE:
        from paper_2407_13996_amd import build as B
        if _DIR is None:
            _DIR = tempfile.mkdtemp(prefix="sgdrc_asm_")
        out = os.path.join(_DIR, os.path.basename(path) + ".s")
        flags = [f for f in B.CFLAGS if f not in ("-fPIC", "-Wall")]
        cmd = [B.HIPCC, *flags, "--cuda-device-only", "-S", path, "-o", out]
        subprocess.run(cmd, check=True, capture_output=True)
        _CACHE[path] = open(out).read()
    return _CACHE[path]


def demangle(names):
    """Demangled C++ names (llvm-cxxfilt), in order."""
    tool = "/opt/rocm/llvm/bin/llvm-cxxfilt"
    if not os.path.exists(tool):
        tool = "c++filt"
    r = subprocess.run([tool], input="\n".join(names), capture_output=True, text=True, check=True)
    return r.stdout.strip().split("\n")


def kernel_resources(asm: str):
    """{demangled kernel name: {vgpr, agpr, sgpr, vgpr_spill, sgpr_spill, lds, scratch}}
    from the amdhsa.kernels metadata of an assembly listing."""
    meta = asm[asm.find("amdhsa.kernels:"):]
    items = re.split(r"\n  - ", meta)[1:]
    keys = {".vgpr_count": "vgpr", ".agpr_count": "agpr", ".sgpr_count": "sgpr",
            ".vgpr_spill_count": "vgpr_spill", ".sgpr_spill_count": "sgpr_spill",
            ".group_segment_fixed_size": "lds", ".private_segment_fixed_size": "scratch"}
    recs, names = [], []
    for it in items:
        rec = {}
        for line in ("  " + it).split("\n"):
            m = re.match(r"^\s+(\.\w+):\s+(\S+)", line)
            if m and m.group(1) in keys:
                rec[keys[m.group(1)]] = int(m.group(2))
            m = re.match(r"^\s+\.name:\s+(\S+)", line)
            if m and "name" not in rec:
                rec["name"] = m.group(1)
        if "name" in rec and "vgpr" in rec:
            recs.append(rec)
            names.append(rec["name"])
    out = {}
    for rec, nm in zip(recs, demangle(names)):
        rec.pop("name")
        out[nm.split("(")[0].replace("void ", "")] = rec
    return out
