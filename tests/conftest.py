import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: full-size cases")


def load_golden(name):
    """Parse a tests/golden key = value fixture (floats, or comma lists)."""
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, v = (s.strip() for s in line.split("=", 1))
            vals = [float(x) for x in v.split(",")]
            out[k] = vals[0] if len(vals) == 1 else vals
    return out


@pytest.fixture(scope="session")
def appendix():
    return load_golden("appendix_counterexample.txt")
