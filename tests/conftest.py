import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP path")


def pytest_collection_modifyitems(config, items):
    # GPU tests fail loudly on a machine without a GPU rather than skipping,
    # unless they were deselected with -m "not gpu".
    pass
