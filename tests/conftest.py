import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def pytest_terminal_summary(terminalreporter):
    """Max elementwise and normwise relative error of every bf16 output the
    GPU parity tests compared with the oracle's fp64 value."""
    try:
        from helpers import ERROR_REPORT
    except ImportError:
        return
    if not ERROR_REPORT:
        return
    tr = terminalreporter
    tr.section("bf16 output vs oracle (fp64): relative errors")
    tr.write_line(f"{len(ERROR_REPORT)} outputs compared; the 24 with the largest elementwise error:")
    tr.write_line(f"{'case':44s} {'M,K,N':>20s} {'scales':>8s} {'max elementwise':>16s} {'normwise':>10s}")
    for label, shape, mode, mx, nw in sorted(ERROR_REPORT, key=lambda r: -r[3])[:24]:
        tr.write_line(f"{label[:44]:44s} {','.join(map(str, shape)):>20s} {mode:>8s} {mx:16.3e} {nw:10.3e}")
    worst = {m: max((r[3] for r in ERROR_REPORT if r[2] == m), default=0.0) for m in ("channel", "group")}
    tr.write_line(f"worst max elementwise: channel {worst['channel']:.3e}, group {worst['group']:.3e}")
