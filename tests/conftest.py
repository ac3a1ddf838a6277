import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


_SCAN_CACHE = {}


@pytest.fixture(scope="session")
def scan_cache():
    """Generated scans are deterministic; generate each (config, frame) once."""
    from synth import CONFIGS, gen_scan

    def get(ci, frame=0):
        key = (ci, frame)
        if key not in _SCAN_CACHE:
            _SCAN_CACHE[key] = gen_scan(CONFIGS[ci], frame)
        return _SCAN_CACHE[key]

    return get
