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
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size oracle comparison (tens of seconds on the host)")


def pytest_collection_modifyitems(config, items):
    # GPU tests cannot run without a device; skip them with a clear reason instead of failing.
    try:
        import torch
        have_gpu = torch.cuda.is_available()
    except Exception:
        have_gpu = False
    if have_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    # worst parity errors per checked workload (collected by tests/parity.py)
    try:
        import parity
    except Exception:
        return
    if parity.SUMMARY:
        terminalreporter.write_sep("-", "parity against the oracle")
        for line in parity.SUMMARY:
            terminalreporter.write_line(line)
