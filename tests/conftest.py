import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libcats")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(scope="session", params=["f32", "f64"])
def oracle_any(request):
    import oracle

    return oracle.load(request.param)


@pytest.fixture(scope="session")
def oracle32():
    import oracle

    return oracle.load("f32")


@pytest.fixture(scope="session")
def oracle64():
    import oracle

    return oracle.load("f64")
