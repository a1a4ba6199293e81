"""Shared pytest configuration: the ``gpu`` marker and cached inputs."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


_BATCHES = {}


def cached_config(n):
    """Workload ``n`` drawn once per test session."""
    from paper_2501_12162_amd.workload import make_config
    if n not in _BATCHES:
        _BATCHES[n] = make_config(n)
    return _BATCHES[n]
