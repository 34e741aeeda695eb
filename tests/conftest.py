import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU check")


@pytest.fixture(scope="session")
def toy():
    """Four tokens small enough to evaluate every equation by hand."""
    import numpy as np
    return dict(
        F=np.array([[1.0, 0.0], [1.0, 0.0], [0.0, 1.0], [1.0, 1.0]]),
        X=np.array([[0, 0, 0], [1, 0, 0], [0, 2, 0], [2, 2, 0]], np.float32),
        tau=np.array([0, 1, 1, 2], np.int32),
        v=np.full(4, 0.25, np.float32),
    )
