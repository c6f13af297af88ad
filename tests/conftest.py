"""Shared test set-up: the gpu marker, and in-tree builds of the oracle and of
librfq when (and only when) nothing is built yet."""
import os
import sys

import pytest

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if REPO not in sys.path:
    sys.path.insert(0, REPO)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def pytest_sessionstart(session):
    import oracle
    if not os.path.exists(oracle.LIB):
        oracle.build()
    from paper_2608_26581_amd import build as rfq_build
    if not os.path.exists(rfq_build.LIB_PATH):
        rfq_build.build()


@pytest.fixture(scope="session")
def orc():
    import oracle
    return oracle.default()
