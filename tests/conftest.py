import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libmsda.so")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """One line per full-size parity case: normwise / 99.9th-percentile element-wise error of
    every output (the tolerances are in tests/gpu_util.py)."""
    gpu_util = sys.modules.get("gpu_util")
    lines = gpu_util.summary_lines() if gpu_util and getattr(gpu_util, "SUMMARY", None) else []
    if lines:
        terminalreporter.write_sep("-", "full-size parity, normwise/p99.9 elementwise error (tol: out 1e-5/1e-4 fp32, "
                                        "1e-3 fp16; gv 1e-4; other grads 1e-3)")
        for line in lines:
            terminalreporter.write_line(line)
