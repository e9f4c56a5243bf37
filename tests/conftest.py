import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Table of the parity configurations run: rows compared, largest row-wise
    relative logit error, oracle near-ties under tol and 2 tol, and token
    mismatches at near-ties (the only mismatches the rule allows)."""
    pu = sys.modules.get("tests.parity_util")
    rec = getattr(pu, "RECORDED", None) if pu else None
    if not rec:
        return
    tr = terminalreporter
    tr.write_sep("-", "parity statistics")
    tr.write_line("| configuration | rows | max rel err | near (< tol) | near (< 2 tol) | mismatches at near-ties |")
    tr.write_line("|---|---|---|---|---|---|")
    for name, s in rec.items():
        tr.write_line(f"| {name} | {s['rows']} | {s['max_rel']:.2e} | {s['near']} | {s['near2']} | "
                      f"{s['mismatch_near']} |")
    path = os.environ.get("KF_PARITY_STATS")
    if path:
        with open(path, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
