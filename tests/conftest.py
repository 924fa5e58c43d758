"""Shared pytest configuration.

Markers:
  gpu -- needs an MI355X (gfx950) and the built HIP library; run with
         ``-m gpu``.  Everything else runs on the CPU.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X GPU and the built HIP library")


@pytest.fixture(scope="session")
def cuda_device():
    """The GPU the parity tests run on.  A GPU test that finds no GPU fails
    (it does not skip): the suite marked gpu is only run where one exists."""
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    return torch.device("cuda:0")


@pytest.fixture(params=["default", "dynamic"])
def schedule(request, monkeypatch):
    """Run a test under the library's own schedule and with the dynamic share
    wherever the planner allows one (DECODE_ATTN_DYNAMIC_MIN_UNITS=0): small
    caches are otherwise wholly static, and the dynamic units, visits and
    claims must stay covered by small, oracle-checked shapes too."""
    if request.param == "dynamic":
        monkeypatch.setenv("DECODE_ATTN_DYNAMIC_MIN_UNITS", "0")
    else:
        monkeypatch.delenv("DECODE_ATTN_DYNAMIC_MIN_UNITS", raising=False)
    return request.param
