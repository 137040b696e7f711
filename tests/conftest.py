import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """Parity margins of the session: per test file, the number of checks
    and the largest observed error as a fraction of its bar."""
    try:
        from _gpu import MARGINS
    except Exception:
        return
    if not MARGINS:
        return
    per = {}
    for test, name, err, tol in MARGINS:
        f = test.split("::")[0]
        n, worst, where = per.get(f, (0, -1.0, ""))
        r = err / tol
        per[f] = (n + 1, r, f"{test} {name}") if r > worst else (n + 1, worst, where)
    terminalreporter.write_sep("-", "parity margins (largest error / bar per file)")
    for f, (n, worst, where) in sorted(per.items()):
        terminalreporter.write_line(f"{f}: {n} checks, worst {worst:.3f} of the bar ({where})")
