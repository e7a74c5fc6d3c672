import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)

from parity_record import MARGINS as _MARGINS  # noqa: E402


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    if not _MARGINS:
        return
    tr = terminalreporter
    tr.section("parity margins (worst slice; max = inf-norm relative, rms = RMS relative)")
    tr.write_line("%-34s %-7s %6s %10s %10s %8s %7s" % ("case", "tensor", "slices", "max_rel", "rms_rel", "tol",
                                                      "margin"))
    for m in _MARGINS:
        tr.write_line("%-34s %-7s %6d %10.3e %10.3e %8.0e %6.1fx" % (
            m["case"][:34], m["tensor"], m["slices"], m["max_rel"], m["rms_rel"], m["tol"],
            m["tol"] / m["max_rel"] if m["max_rel"] > 0 else float("inf")))
    out_dir = os.path.join(ROOT, "gpurun_out")
    if os.path.isdir(out_dir):
        try:
            with open(os.path.join(out_dir, "parity_margins.json"), "w") as f:
                json.dump(_MARGINS, f, indent=1)
        except OSError:
            pass


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def gpu():
    if not gpu_available():
        pytest.skip("no GPU visible")
    import torch
    return torch.device("cuda:0")
