import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


@pytest.fixture(scope="session")
def rng():
    import numpy as np
    return np.random.default_rng(20250100692)


def pytest_sessionfinish(session, exitstatus):
    """Write every parity check's rel-L2 (test, output, error, tolerance) as JSON
    lines into the file named by SSM_PARITY_RECORD, if set."""
    path = os.environ.get("SSM_PARITY_RECORD")
    if not path:
        return
    try:
        from gpu_helpers import RECORD
    except ImportError:
        return
    import json
    os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
    with open(path, "w") as f:
        for test, name, err, tol in RECORD:
            f.write(json.dumps({"test": test, "output": name, "rel_l2": err, "tol": tol}) + "\n")
