import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workload case (minutes of host work)")


def pytest_terminal_summary(terminalreporter):
    """The plain metric of every GEMM parity check this session made
    (tests/gpu_util.py REPORT): max |err| / sum |ab| without the matrix
    instruction's truncation allowance, and the fraction of entries above
    1e-5. Also written as JSON to $PURO_PARITY_REPORT when that is set."""
    mod = sys.modules.get("gpu_util")
    if mod is None or not mod.REPORT:
        return
    import json
    rep = mod.REPORT
    tr = terminalreporter
    tr.section("GEMM parity, plain metric max|err|/sum|ab| (bound %g)" % mod.TOL)
    for r in rep:
        tr.write_line("%-60s %4s %9d entries  max %.3e  above bound %.2e%s" % (
            r["what"][:60], r["kind"], r["entries"], r["max_rel"], r["plain_excess"],
            "  (asserted)" if r["strict"] else ""))
    path = os.environ.get("PURO_PARITY_REPORT")
    if path:
        with open(path, "w") as f:
            json.dump(rep, f, indent=1)
