"""The driver's smoke check, __graft_entry__.smoke(), run as a GPU test: one small forward of
the hot path on cuda:0 against the oracle, through the same calls the driver makes."""

import os
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_smoke_entry_point():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    sys.path.insert(0, ROOT)
    import __graft_entry__
    __graft_entry__.smoke()
