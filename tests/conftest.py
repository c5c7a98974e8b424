"""Shared pytest configuration.

Markers:
  gpu   needs an MI355X (gfx950); every such test calls the GPU library through its C ABI.
  slow  long-running (full-size parameter sets); still part of the default run.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU (gfx950)")
    config.addinivalue_line("markers", "slow: long-running full-size case")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    oracle.build()
    return oracle
