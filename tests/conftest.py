import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large synthetic workload")


def read_golden(name):
    """Parse a ``key v1 v2 ...`` fixture under tests/golden (``#`` starts a comment)."""
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *vals = line.split()
            out[key] = vals
    return out


@pytest.fixture
def golden():
    return read_golden


@pytest.fixture(scope="session", autouse=True)
def _built_libraries():
    """Build the oracle and libdigest.so only if nothing is built yet."""
    import oracle
    oracle.build()
    from paper_2206_00057_amd import build as B
    if not os.path.exists(B.LIB):
        B.build()
