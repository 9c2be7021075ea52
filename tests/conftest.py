import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP C-ABI)")


def load_golden(name):
    """Parse a fixture under tests/golden: '#' comments, then name/shape and value lines."""
    path = os.path.join(ROOT, "tests", "golden", name)
    lines = [l.strip() for l in open(path) if l.strip() and not l.lstrip().startswith("#")]
    out = {}
    for i in range(0, len(lines), 2):
        key, shape = lines[i].split()
        shape = tuple(int(s) for s in shape.split(","))
        vals = np.array([float(v) for v in lines[i + 1].split(",")], dtype=np.float64)
        out[key] = vals.reshape(shape)
    return out


@pytest.fixture
def golden():
    return load_golden
