import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_collection_modifyitems(config, items):
    # GPU tests must run only where a GPU is present; on a CPU machine they are
    # deselected by `-m "not gpu"`.  When run anyway without a GPU they fail
    # loudly instead of silently passing on some fallback.
    pass
