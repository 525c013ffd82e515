import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """Error statistics of the full-size parity cases (tests/parity.py STATS)."""
    from tests import parity
    if not parity.STATS:
        return
    tr = terminalreporter
    tr.write_sep("-", "full-size parity: max|gpu-ref|/max|ref|, element-wise rel. err p99.9 / max")
    for case, name, e, p999, emax in parity.STATS:
        tr.write_line("%-22s %-18s %.2e  %.2e / %.2e" % (case, name, e, p999, emax))
