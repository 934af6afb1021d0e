import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def gpu_available():
    import torch
    return torch.cuda.is_available()


def pytest_terminal_summary(terminalreporter):
    """Worst bf16 output errors per test (raw max-abs, raw where |y| < 4,
    excess beyond half a bf16 step where |y| >= 4, rel-L2), so the margin
    under the 2e-2 / 1e-2 bars is visible in the test log."""
    pu = sys.modules.get("parity_util")
    rows = getattr(pu, "BF16_REPORT", None) if pu else None
    if not rows:
        return
    worst = {}
    for test, where, raw, raw_small, excess, rel in rows:
        w = worst.setdefault(test, [0.0, 0.0, float("-inf"), 0.0, 0])
        w[0], w[1], w[2], w[3] = max(w[0], raw), max(w[1], raw_small), max(w[2], excess), max(w[3], rel)
        w[4] += 1
    tr = terminalreporter
    tr.write_sep("-", "bf16 output margins (bars: max-abs 2e-2, rel-L2 1e-2)")
    tr.write_line(f"{'checks':>6} {'raw':>9} {'raw|y|<4':>9} {'excess':>9} {'relL2':>9}  test")
    for test, (raw, raw_small, excess, rel, n) in sorted(worst.items()):
        ex = f"{excess:9.2e}" if excess != float("-inf") else f"{'-':>9}"
        tr.write_line(f"{n:6d} {raw:9.2e} {raw_small:9.2e} {ex} {rel:9.2e}  {test}")
