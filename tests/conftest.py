import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


import pytest


@pytest.fixture(scope="session")
def built_lib():
    """Path of the HIP library; built once if nothing is built yet."""
    from paper_2607_19547_amd import binding, build
    if not os.path.exists(binding.LIB_PATH):
        build.build()
    return binding.LIB_PATH
