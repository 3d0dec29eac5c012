import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


def pytest_terminal_summary(terminalreporter):
    """Decision counts of every GPU-vs-oracle comparison (parity.py)."""
    mod = sys.modules.get("parity")
    if mod is None or not mod.REPORT:
        return
    tr = terminalreporter
    tr.section("acceptance decisions compared")
    tr.write_line("test | checked vs oracle | flagged (margin/straddle) | accepted drafts checked | "
                  "self-checked on GPU logits | self margin")
    for name, checked, flagged, accepted, sc, sm in mod.REPORT:
        tr.write_line(f"{name} | {checked} | {flagged} | {accepted} | {sc if sc is not None else '-'} | "
                      f"{sm if sm is not None else '-'}")
