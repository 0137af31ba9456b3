import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Per-comparison parity reports (exempt / swapped node counts, how many nodes the
    bands admit, the largest errors), printed whatever the verbosity."""
    parity = sys.modules.get("parity")
    reports = getattr(parity, "REPORTS", None)
    if not reports:
        return
    tr = terminalreporter
    tr.write_sep("=", "parity reports (GPU vs fp64 oracle)")
    tr.write_line(f"{'case':44s} {'nodes':>6s} {'exempt':>6s} {'admis.':>6s} {'swap':>5s} "
                  f"{'h rel':>9s} {'r rel':>9s} {'mass err':>9s} {'gate err':>9s}")
    for r in reports:
        tr.write_line(f"{r['label'][:44]:44s} {r['n']:6d} {r['exempt']:6d} {r['admissible']:6d} "
                      f"{r['swapped']:5d} {r['h_rel_max']:9.2e} {r['r_rel_max']:9.2e} "
                      f"{r['mass_err_max']:9.2e} {r['gate_err_max']:9.2e}")
