import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """The per-tensor parity margins of the GPU tests that ran: printed (also
    under -q) and written to gpurun_out/parity_margins.json."""
    try:
        from helpers import MARGINS
    except ImportError:
        return
    if not MARGINS:
        return
    tr = terminalreporter
    tr.section("parity margins (error / bound per output tensor, worst first)")
    for m in sorted(MARGINS, key=lambda m: -m["error"] / m["bound"]):
        fl = "" if m["floor"] is None else f"{m['floor']:.3e}"
        tr.write_line(f"{m['error'] / m['bound']:6.3f}  error {m['error']:.3e}  floor {fl:>9}  "
                      f"bound {m['bound']:.3e}  {'ok' if m['ok'] else 'FAIL'}  {m['test']} {m['tensor']}")
    out = os.path.join(ROOT, "gpurun_out")
    try:
        os.makedirs(out, exist_ok=True)
        with open(os.path.join(out, "parity_margins.json"), "w") as f:
            json.dump(MARGINS, f, indent=0)
    except OSError:
        pass
