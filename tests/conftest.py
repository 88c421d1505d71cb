import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def pytest_collection_modifyitems(config, items):
    """GPU tests are skipped (not failed) when no GPU is visible."""
    try:
        import torch
        has_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        has_gpu = False
    if has_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(skip)


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Counts of the end-to-end parity checks (GPU error against the exact
    oracle, next to the CPU bf16-storage emulation's) for the run's log."""
    try:
        from parity import summary_lines
    except Exception:  # pragma: no cover
        return
    lines = summary_lines()
    if lines:
        terminalreporter.write_sep("-", "end-to-end parity against the exact oracle")
        for line in lines:
            terminalreporter.write_line(line)
