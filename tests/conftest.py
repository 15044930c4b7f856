import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """Print the Adam comparison counts of the whole-partition checks: per
    array, the elements compared, equal bit for bit, passing the strict
    rule, and passing only the derived bound."""
    parity = sys.modules.get("parity")
    counts = getattr(parity, "ADAM_COUNTS", None)
    if not counts:
        return
    tr = terminalreporter
    tr.section("Adam parity counts (n / bitwise / strict / derived bound only)")
    for what, c in counts:
        tr.write_line(what)
        for name, k in c.items():
            tr.write_line("  %-10s %11d %11d %11d %9d (%.2e)" % (
                name, k["n"], k["bitwise"], k["strict"], k["relaxed_only"],
                k["relaxed_only"] / max(1, k["n"])))
