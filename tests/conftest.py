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
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_sessionfinish(session, exitstatus):
    """Write the per-tensor parity errors of this session (GPU tests only)."""
    import parity_log

    rows = parity_log.rows()
    if not rows:
        return
    out = os.path.join(ROOT, "gpurun_out")
    os.makedirs(out, exist_ok=True)
    with open(os.path.join(out, "parity_margins.tsv"), "w") as f:
        f.write("case\ttensor\tmax_rel_err\tbound\tbound/err\n")
        for case, tensor, err, tol in rows:
            ratio = tol / err if err > 0 else float("inf")
            f.write(f"{case}\t{tensor}\t{err:.3e}\t{tol:.0e}\t{ratio:.1f}\n")
