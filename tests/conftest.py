import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
TESTS = os.path.dirname(os.path.abspath(__file__))
if TESTS not in sys.path:
    sys.path.insert(0, TESTS)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


GOLDEN = os.path.join(TESTS, "golden")


def golden_path(name: str) -> str:
    return os.path.join(GOLDEN, name)


def read_kv(name: str) -> dict:
    """key = value lines of a golden file (values split on whitespace)."""
    out = {}
    with open(golden_path(name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if "=" in line and not line.startswith("step"):
                k, v = (x.strip() for x in line.split("=", 1))
                out[k] = v
    return out


@pytest.fixture(scope="session")
def oracle_lib():
    from oracle import oracle
    oracle.build()
    return oracle
