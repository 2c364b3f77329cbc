import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


@pytest.fixture(scope="session")
def tiny():
    import numpy as np  # noqa: F401
    import oracle
    import synth
    w = synth.WORKLOADS["tiny"]
    blob = synth.make_weights(w.model, 0)
    return w, blob, oracle.Model(w.model, blob)
