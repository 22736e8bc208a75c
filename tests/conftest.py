import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP C-ABI library)")
    config.addinivalue_line("markers", "slow: long-running (full-size shapes)")


@pytest.fixture(scope="session")
def tiny_weights():
    """Oracle weight views (bf16-boundary) of the tiny workloads, generated once per session."""
    import synth
    from oracle.numerics import WeightView
    cache = {}

    def get(key):
        if key not in cache:
            w = synth.WORKLOADS[key]
            cache[key] = (w, synth.make_weights(w.geom))
        w, stored = cache[key]
        return w, stored, WeightView(stored)

    return get
