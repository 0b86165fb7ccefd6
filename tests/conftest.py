import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def pytest_terminal_summary(terminalreporter):
    """Achieved parity errors of the GPU tests that ran (worst per test and
    quantity, beside the bound each was held to)."""
    try:
        import gpu_harness as H
    except Exception:
        return
    if not H.ERRORS:
        return
    tr = terminalreporter
    tr.section("achieved parity errors (worst value / bound)")
    for (test, q), (v, b, where) in sorted(H.ERRORS.items()):
        tr.write_line(f"{test:60s} {q:22s} {v:10.3e} / {b:9.2e}  {where}")
    out = os.environ.get("PARITY_ERRORS_JSON")
    if out:
        import json
        with open(out, "w") as fh:
            json.dump([{"test": t, "quantity": q, "value": v, "bound": b, "where": wh}
                       for (t, q), (v, b, wh) in sorted(H.ERRORS.items())], fh, indent=1)
