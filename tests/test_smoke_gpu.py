"""The package's smoke entry point (one small pass of the whole hot path on
cuda:0, checked against the oracle) run as a GPU test."""
import pytest
import torch

import __graft_entry__ as entry

pytestmark = pytest.mark.gpu


def test_smoke():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    entry.smoke()
