import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session", autouse=True)
def _built_helpers():
    """The oracle and the input generator are small gcc builds; build them
    if absent (the device library is built by __graft_entry__.build())."""
    import oracle
    import synth
    oracle.build()
    synth.build()
    yield
