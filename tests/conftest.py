import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle


def pytest_terminal_summary(terminalreporter):
    """Report the GEMV parity tests' observed error against the bound of the
    kernel's summation tree (largest |y - ref| / sum|W x| per case)."""
    log = None
    for name, mod in list(sys.modules.items()):
        if name.rsplit(".", 1)[-1] == "test_gpu_parity":
            log = getattr(mod, "ERR_LOG", None)
    if not log:
        return
    tr = terminalreporter
    worst = max(r / (2 * d * 2.0 ** -24) for r, d in log.values())
    tr.write_line(f"GEMV error: {len(log)} checks; largest observed error / bound = {worst:.3f}")
    for (M, K, B, wd, xd, n, tag), (r, d) in sorted(log.items(), key=lambda kv: str(kv[0])):
        tr.write_line(f"  {M}x{K} B={B} w={wd} x={xd} cus={n} {tag}: max|err|/sum|Wx| = {r:.3g}, "
                      f"bound {2 * d * 2.0 ** -24:.3g} (depth {d})")
