import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    # another build of the same sources, e.g. the sanitizer builds that
    # tests/test_sanitizers.py makes (test runs only)
    if os.environ.get("SPIRE_TEST_LIB"):
        from paper_2504_06419_amd import spire
        spire.LIB_PATH = os.environ["SPIRE_TEST_LIB"]
    if os.environ.get("SPIRE_TEST_ORACLE_LIB"):
        from oracle import oracle as O
        O.LIB = os.environ["SPIRE_TEST_ORACLE_LIB"]


def pytest_collection_modifyitems(config, items):
    """Skip GPU tests cleanly where no GPU is visible (collection still works)."""
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
