import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """The worst attention error of every parity replay that ran."""
    mod = sys.modules.get("_parity")
    if mod is None or not getattr(mod, "WORST", None):
        return
    terminalreporter.write_line("attention parity, worst |gpu - oracle| per replay (elementwise bar "
                                "1e-3 + 2e-3 |ref|; bf16 output adds 2^-8 |ref|):")
    for test, (worst, n, out) in sorted(mod.WORST.items()):
        terminalreporter.write_line(f"  {test}: {worst:.3g} over {n} outputs ({out} output)")
