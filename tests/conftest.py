import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def pytest_terminal_summary(terminalreporter):
    """How often the index-set comparisons of this session met near-tie swaps
    (only if a test used the comparison)."""
    helpers = sys.modules.get("helpers")
    stats = getattr(helpers, "SWAP_STATS", None)
    if stats and stats["units"]:
        terminalreporter.write_line(
            f"index sets compared: {stats['units']} units, {stats['swapped_units']} with "
            f"tolerated near-tie swaps (at most {stats['max_entries']} entries in one unit, "
            f"largest gap {stats['max_gap_rel']:.2e} of |tau|)")
