"""The round-trip check __graft_entry__.smoke() runs (a small network on the
GPU against the oracle), kept under test so that it cannot break unnoticed."""
import os
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_smoke_entry_point():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sys.path.insert(0, ROOT)
    import __graft_entry__
    __graft_entry__.smoke()
