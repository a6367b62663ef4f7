"""Shared pytest configuration: registers the `gpu` marker and puts the repo root on sys.path."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_terminal_summary(terminalreporter):
    """Normwise and elementwise errors of the whole-path parity tests that ran
    (bounds: normwise 1e-5 in fp32, 2e-2 in bf16; the elementwise figure is
    reported, not bounded)."""
    try:
        from gpu_helpers import PARITY_LOG
    except ImportError:
        return
    if not PARITY_LOG:
        return
    tr = terminalreporter
    tr.write_sep("-", "whole-path parity: max|g-o|/max|o| (bounded) and max|g-o|/(|o|+1e-3 max|o|) (reported)")
    worst = {}
    for test, tensor, nw, ew in PARITY_LOG:
        w = worst.setdefault(test, [0.0, 0.0, 0])
        w[0], w[1], w[2] = max(w[0], nw), max(w[1], ew), w[2] + 1
    for test, (nw, ew, k) in worst.items():
        tr.write_line(f"{test}: {k} tensors, normwise <= {nw:.2e}, elementwise <= {ew:.2e}")
