import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Print the measured max-relative errors of every GPU parity comparison
    of the session (tolerances: 1e-4 float32, 2e-2 bfloat16), so that the
    margins appear in the run's own output."""
    from tests.harness import MARGINS, TOL
    if not MARGINS:
        return
    tr = terminalreporter
    tr.section("GPU parity margins (max |x - ref| / max |ref| per tensor, fp64 oracle)")
    worst = {}
    for label, dtype, errs in MARGINS:
        k = max(errs, key=errs.get)
        tr.write_line(f"{dtype:4s} {label[:44]:44s} worst {k}={errs[k]:.1e} | " +
                      " ".join(f"{n}={e:.1e}" for n, e in errs.items()))
        if errs[k] > worst.get(dtype, (0.0, ""))[0]:
            worst[dtype] = (errs[k], f"{label} {k}")
    for dtype, (e, where) in worst.items():
        tr.write_line(f"worst {dtype}: {e:.2e} of tolerance {TOL[dtype]:.0e} "
                      f"({e / TOL[dtype]:.1%}) in {where}; {len(MARGINS)} comparisons")
