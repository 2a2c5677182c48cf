import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size case (minutes of CPU oracle time)")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Totals of every parity comparison: elements compared, and failures
    under the plain 1e-4 / 1e-5 rule, per kind of comparison."""
    try:
        from helpers import REPORT
    except ImportError:
        return
    if not REPORT:
        return
    tot = {}
    for _, _, kind, n, plain, bad in REPORT:
        t = tot.setdefault(kind, [0, 0, 0, 0])
        t[0] += 1
        t[1] += n
        t[2] += plain
        t[3] += bad
    w = terminalreporter
    w.write_sep("-", "parity comparisons (plain rule: |gpu-ref| <= 1e-5 + 1e-4|ref|)")
    for kind, (c, n, plain, bad) in sorted(tot.items()):
        w.write_line(f"{kind:9s} comparisons {c:5d}  elements {n:12d}  "
                     f"plain-rule failures {plain:8d}  enforced-rule failures {bad}")
    for tid, name, kind, n, plain, bad in REPORT:
        if plain and kind == "reduction":
            w.write_line(f"  plain-rule failures, sigma rule holds: {tid} {name}: {plain}/{n}")
    path = os.environ.get("SCN_PARITY_REPORT")
    if path:
        with open(path, "w") as f:
            json.dump({"totals": tot, "comparisons": REPORT}, f)
