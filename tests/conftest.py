import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_terminal_summary(terminalreporter):
    """Print every GPU-vs-reference comparison of the run (max-abs, relative L2 and
    the largest reference entry, which shows whether max-abs binds) and, when the
    environment variable PIC_PARITY_SUMMARY names a file, write a copy there."""
    try:
        from tests.gpu_util import RECORDS
    except Exception:  # pragma: no cover
        return
    if not RECORDS:
        return
    lines = [f"{'comparison':64s} {'dtype':5s} {'max_abs':>10s} {'rel_l2':>10s} {'max|ref|':>9s}"]
    for what, ma, rel, peak, dt in RECORDS:
        lines.append(f"{what[:64]:64s} {dt:5s} {ma:10.3e} {rel:10.3e} {peak:9.3g}")
    terminalreporter.write_line("parity records (GPU vs oracle or vs another GPU path):")
    for ln in lines:
        terminalreporter.write_line(ln)
    out = os.environ.get("PIC_PARITY_SUMMARY")
    if out:
        with open(out, "w") as f:
            f.write("\n".join(lines) + "\n")
