import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: full-size parity case")


def rel_err(got, ref):
    """max_i |g_i - r_i| / max(|r_i|, rms(r)): relative with an RMS floor.

    The floor keeps elements that happen to be near zero from dominating;
    a tensor that is entirely zero in the reference is compared absolutely.
    """
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(ref * ref)))
    denom = np.maximum(np.abs(ref), rms)
    denom = np.where(denom == 0.0, 1.0, denom)
    return float(np.max(np.abs(got - ref) / denom))


@pytest.fixture
def rng():
    return np.random.default_rng(1234)
