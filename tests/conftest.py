import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import seeded_inputs as si  # noqa: E402


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size case (minutes of CPU oracle work)")


def weights_f64(w: dict, dtype: str) -> dict:
    """{stream: {tensor: storage}} -> same structure in float64."""
    return {s: {t: si.as_f64(a, dtype) for t, a in ws.items()} for s, ws in w.items()}


@pytest.fixture
def rng():
    return np.random.default_rng(1234)
