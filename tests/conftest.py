import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def oracle_lib():
    import oracle
    oracle.build(force=False)
    return oracle


def read_golden(name):
    """Parse a tests/golden/*.txt file: comment lines start with '#'."""
    path = os.path.join(ROOT, "tests", "golden", name)
    recs = []
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            recs.append(line.split())
    return recs


def kv(fields):
    """key=value fields of a golden record -> dict (other fields are ignored)."""
    out = {}
    for f in fields:
        if "=" in f:
            a, b = f.split("=", 1)
            out[a] = b
    return out
