import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: CPU test that takes more than a few seconds")


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")


def _quantiles(x):
    import numpy as np

    x = np.sort(np.asarray(x, np.float64).ravel())
    if x.size == 0:
        return None
    return {"max": float(x[-1]), "p99.9": float(x[int(0.999 * (x.size - 1))]),
            "median": float(x[x.size // 2])}


@pytest.fixture
def parity_log():
    """Record plain relative errors (max, p99.9, median) of a parity test: printed, and
    appended as one JSON line to the file named by $ERC_PARITY_LOG when it is set."""
    import json

    import numpy as np

    def log(case, **pairs):
        rec = {"case": case}
        for key, (got, want) in pairs.items():
            got = np.asarray(got, np.float64)
            want = np.asarray(want, np.float64)
            nz = want != 0
            rec[key] = _quantiles(np.abs(got - want)[nz] / np.abs(want[nz]))
        print(json.dumps(rec))
        path = os.environ.get("ERC_PARITY_LOG")
        if path:
            with open(path, "a") as f:
                f.write(json.dumps(rec) + "\n")
        return rec

    return log
