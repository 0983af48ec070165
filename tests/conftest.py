import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running parity case")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Parity numbers of the GPU checks: the full-size workloads one by one,
    then the worst case per dtype over every check of the session."""
    try:
        from tests import gpu_util
    except Exception:
        return
    recs = getattr(gpu_util, "RECORDS", [])
    if not recs:
        return
    tr = terminalreporter
    tr.write_line("parity: raw = max|y - y_ref| / rms(y_ref) with output rounding, "
                  "excess = beyond output rounding (the tolerance's quantity)")
    for what, name, raw, e, tol, full in recs:
        if full:
            tr.write_line(f"  [full size] {what}: raw {raw:.3e}, excess {e:.3e} <= {tol:.0e} ({name})")
    for name in ("fp32", "bf16"):
        rs = [r for r in recs if r[1] == name]
        if rs:
            worst = max(rs, key=lambda r: r[3] / r[4])
            tr.write_line(f"  {name}: {len(rs)} checks, largest raw {max(r[2] for r in rs):.3e}, "
                          f"largest excess {worst[3]:.3e} of limit {worst[4]:.0e} ({worst[0]})")
