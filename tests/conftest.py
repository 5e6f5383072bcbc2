import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def pytest_terminal_summary(terminalreporter):
    """The literal max-abs error of every bf16 GPU-vs-oracle comparison the
    session made, with those above 2e-2 marked: the gate adds the output's own
    bf16 rounding (2^-8 |ref|), so these are visible rather than silent."""
    from tests import parity
    if not parity.RECORD:
        return
    tr = terminalreporter
    over = [r for r in parity.RECORD if r[1] > parity.ATOL_BF16]
    tr.write_line(f"bf16 parity: {len(parity.RECORD)} comparisons; literal max|gpu - ref| "
                  f"above {parity.ATOL_BF16:g} in {len(over)} (each within 2e-2 + 2^-8 |ref|)")
    worst = max(parity.RECORD, key=lambda r: r[1])
    tr.write_line(f"  largest: {worst[0]}: max_abs={worst[1]:.3e} max|ref|={worst[4]:.3e}")
    for what, max_abs, excess, rel, ref_max in over:
        tr.write_line(f"  > 2e-2: {what}: max_abs={max_abs:.3e} beyond_rounding={excess:.3e} "
                      f"rel_fro={rel:.3e} max|ref|={ref_max:.3e}")
