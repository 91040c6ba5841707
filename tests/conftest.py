import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def random_profile(M: int, seed: int, alpha: float = 1.0, talpha: float = 1.0):
    """A profile with random emissions AND random per-node transitions, so
    that a transposed or mis-indexed transition changes some score.  Small
    alpha / talpha give peaked emissions / transitions, which make insert
    runs, delete runs and multi-hit (J) paths win often."""
    from synth import BACKGROUND, Profile
    rng = np.random.default_rng(seed)
    match = rng.dirichlet(np.full(20, alpha), size=M)
    insert = rng.dirichlet(np.full(20, alpha), size=max(M - 1, 0))
    tr = np.zeros((max(M - 1, 0), 7))
    for k in range(M - 1):
        tr[k, 0:3] = rng.dirichlet(np.array([2.0, 1.0, 1.0]) * talpha)
        tr[k, 3:5] = rng.dirichlet(np.array([1.0, 1.0]) * talpha)
        tr[k, 5:7] = rng.dirichlet(np.array([1.0, 1.0]) * talpha)
    tr[:, 0:3] = (tr[:, 0:3] + 1e-3) / (1 + 3e-3)
    tr[:, 3:5] = (tr[:, 3:5] + 1e-3) / (1 + 2e-3)
    tr[:, 5:7] = (tr[:, 5:7] + 1e-3) / (1 + 2e-3)
    match = (match + 1e-3) / (1 + 20e-3)
    insert = (insert + 1e-3) / (1 + 20e-3)
    return Profile(M, BACKGROUND.copy(), match, insert, tr)


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    oracle.lib()
    return oracle
