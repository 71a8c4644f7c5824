import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libtg.so")
    config.addinivalue_line("markers", "slow: full-size workload (minutes)")


def u16(t):
    """torch bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    import torch
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view("uint16")


@pytest.fixture
def to_u16():
    return u16
