import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def _print_case(item):
    # name the case before any GPU work starts, so a crash still says which
    print(f"\n[case] {item.nodeid}", flush=True)


def pytest_runtest_setup(item):
    if item.get_closest_marker("gpu") is not None:
        _print_case(item)


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    oracle.build()
    return oracle
