import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP library)")
    config.addinivalue_line("markers", "slow: full-size case (minutes)")


def pytest_collection_modifyitems(config, items):
    # GPU tests cannot run on a host without a GPU; skip them loudly there
    # instead of failing, so `-m "not gpu"` and plain runs stay meaningful.
    try:
        import torch
        have_gpu = torch.cuda.is_available()
    except Exception:  # pragma: no cover
        have_gpu = False
    if have_gpu:
        return
    skip = pytest.mark.skip(reason="no GPU visible")
    for item in items:
        if "gpu" in item.keywords:
            item.add_marker(skip)


@pytest.fixture(scope="session")
def parrot_lib():
    """The built C library (built in-tree first if it is missing)."""
    from paper_2405_19888_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2405_19888_amd.build import build
        build()
    return binding.load_library()
