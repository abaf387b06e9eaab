import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a GPU (MI355X) and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU-side runs")


def _ensure_built():
    """Build the CPU-side helpers (oracle, generator) only when nothing is built."""
    import oracle
    import workloads
    oracle.build(force=False)
    workloads.build(force=False)


_ensure_built()
