import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
for path in (ROOT, HERE):
    if path not in sys.path:
        sys.path.insert(0, path)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: full-size case (seconds of oracle time)")


def pytest_collection_modifyitems(config, items):
    # Tests that need a GPU are skipped, not failed, where none is visible.
    have_gpu = None
    for item in items:
        if "gpu" in item.keywords:
            if have_gpu is None:
                import torch
                have_gpu = torch.cuda.is_available()
            if not have_gpu:
                item.add_marker(pytest.mark.skip(reason="no GPU visible"))


@pytest.fixture(scope="session")
def xcheck_libs(tmp_path_factory):
    """Independent open-source Philox engines built for the host (test-only)."""
    import engines
    return engines.build(tmp_path_factory.mktemp("xcheck"))
