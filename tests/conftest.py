import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """The elementwise diagnostic |g - r| / (|r| + rms(r)) of the parity
    checks: the worst value per test and dtype (reported, not a criterion;
    the pass criterion is the normwise error)."""
    mod = sys.modules.get("tests.gpu_util")
    diag = getattr(mod, "DIAG", None)
    if not diag:
        return
    tr = terminalreporter
    tr.section("elementwise diagnostic |g-r|/(|r|+rms(r)), worst per test")
    for (test, dtype), (d, what) in sorted(diag.items(), key=lambda kv: -kv[1][0])[:40]:
        tr.write_line(f"{d:10.3e}  {dtype:5s} {test}  ({what})")
    worst = {}
    for (_, dtype), (d, _) in diag.items():
        worst[dtype] = max(worst.get(dtype, 0.0), d)
    tr.write_line("worst per dtype: " + ", ".join(f"{k} {v:.3e}" for k, v in sorted(worst.items())))
