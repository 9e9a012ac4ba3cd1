import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    from oracle import build
    if not os.path.exists(build.LIB):
        build.build()
    return oracle


@pytest.fixture
def tune():
    """Sets kernel-choice overrides of the library for one test
    (``onexn_set_tuning``) and restores the automatic choice afterwards."""
    import paper_2105_14713_amd as onexn
    names = []

    def set_(name, value):
        onexn.set_tuning(name, int(value))
        names.append(name)

    yield set_
    for name in names:
        onexn.set_tuning(name, -1)
