"""Shared pytest configuration.

Tests marked ``gpu`` need an MI355X (gfx950) and the built HIP library; all
other tests run on the CPU only.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an AMD Instinct GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running (full-size workloads)")
    config.addinivalue_line("markers", "cpu_only: hands the library made-up device addresses; "
                                       "skipped where a GPU is visible")


def pytest_collection_modifyitems(config, items):
    # A GPU test on a host without a GPU is skipped; on a GPU host a missing
    # HIP library is an error, raised by the binding itself.
    have_gpu = False
    try:
        import torch
        have_gpu = torch.cuda.is_available()
    except Exception:
        pass
    if have_gpu:
        skip_cpu = pytest.mark.skip(reason="made-up device addresses are tested only without a GPU")
        for it in items:
            if "cpu_only" in it.keywords:
                it.add_marker(skip_cpu)
        return
    skip = pytest.mark.skip(reason="no GPU on this host")
    for it in items:
        if "gpu" in it.keywords:
            it.add_marker(skip)
