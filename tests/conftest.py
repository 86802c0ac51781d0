import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X GPU and the built HIP library")


@pytest.fixture(scope="session")
def tiny_net():
    from synth import NetShape
    return NetShape(in_h=12, in_w=12, in_c=4, ch=(2, 3, 3), hidden=8, num_actions=3)
