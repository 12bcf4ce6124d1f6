import json
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a real MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


@pytest.fixture
def rng():
    return np.random.default_rng(12345)


def lowrank_cell(rng, m, T, d, rank, noise=0.0, decay=1.0):
    """Small random cell with a gapped spectrum (test helper, fp64)."""
    A = rng.standard_normal((T, rank))
    F, _ = np.linalg.qr(rng.standard_normal((d, rank)))
    F = F * (np.arange(1, rank + 1) ** -decay)
    X = np.stack([A @ rng.standard_normal((rank, rank)) @ F.T for _ in range(m)])
    if noise:
        X = X + noise * rng.standard_normal(X.shape)
    return X
