import json
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


# Neurons and images the parity rules exclude (near-threshold neurons,
# ambiguous chained images), gathered per test and written at the end of the
# session to $SPK_PARITY_SUMMARY (default gpurun_out/parity_exclusions.json).
_EXCLUSIONS = []


@pytest.fixture
def near_log(request):
    def log(what, excluded, total):
        _EXCLUSIONS.append({"test": request.node.nodeid, "what": what, "excluded": int(excluded),
                            "total": int(total)})
        print(f"{what}: {int(excluded)} of {int(total)} excluded", flush=True)
    return log


def pytest_sessionfinish(session, exitstatus):
    if not _EXCLUSIONS:
        return
    path = os.environ.get("SPK_PARITY_SUMMARY", os.path.join(ROOT, "gpurun_out", "parity_exclusions.json"))
    os.makedirs(os.path.dirname(path), exist_ok=True)
    summary = {"cases": len(_EXCLUSIONS), "excluded": sum(e["excluded"] for e in _EXCLUSIONS),
               "total": sum(e["total"] for e in _EXCLUSIONS), "records": _EXCLUSIONS}
    with open(path, "w") as f:
        json.dump(summary, f, indent=1)
