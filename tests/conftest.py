"""Shared pytest configuration: the ``gpu`` marker, repository paths and the binding fixture."""
import os
import sys

import pytest

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)
for path in (ROOT, TESTS):
    if path not in sys.path:
        sys.path.insert(0, path)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="module")
def scram():
    """The HIP library's Python binding; loading it raises if the library is missing (no fallback)."""
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1905_10308_amd as scram

    scram.lib()
    return scram
