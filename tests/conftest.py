import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
for p in (ROOT, os.path.join(ROOT, "tests")):
    if p not in sys.path:
        sys.path.insert(0, p)


def pytest_addoption(parser):
    parser.addoption("--pase-lib", default=None,
                     help="load this build of libpase instead of the in-tree one (the sanitizer run "
                          "of the host tests uses the host-only build)")


def pytest_configure(config):
    lib = config.getoption("--pase-lib")
    if lib:
        from paper_2407_04001_amd import pase
        pase.LIB_PATH = lib
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP library on the device)")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(scope="session")
def oracle_lib():
    from oracle import oracle
    oracle.build(force=False)
    return oracle
