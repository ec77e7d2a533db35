import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _gpu_available() -> bool:
    try:
        import torch
        return bool(torch.cuda.is_available())
    except Exception:
        return False


@pytest.fixture(scope="session")
def dp():
    """The Python binding of the C-ABI library, on a machine with a GPU.

    Loading fails loudly (an exception, not a skip) when a GPU is present but
    the built library is missing.
    """
    if not _gpu_available():
        pytest.skip("no GPU visible to torch")
    from paper_2609_20532_amd import dpsgd
    dpsgd.load()
    return dpsgd
