import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def pytest_terminal_summary(terminalreporter):
    """List how many decisions each parity case pinned from the oracle (near
    ties) against the decisions the oracle took freely."""
    try:
        from tests import harness
    except Exception:  # the harness needs numpy and the oracle; nothing to report then
        return
    if not harness.INJECTIONS:
        return
    terminalreporter.write_line("near-tie decisions pinned from the oracle "
                                "(case: boundaries + merges / free decisions):")
    for r in harness.INJECTIONS:
        terminalreporter.write_line(f"  {r['case']}: {r['near_b']} + {r['near_m']} / {r['free']}")
