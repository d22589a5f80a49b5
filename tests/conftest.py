import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: longer CPU test")


GOLDEN = os.path.join(ROOT, "tests", "golden")


@pytest.fixture(scope="session")
def over_by_hand():
    """Cases of tests/golden/over_by_hand.txt: (name, layers [k, 4] front to
    back, result [4]), premultiplied RGBA worked out by hand."""
    import numpy as np
    out = []
    with open(os.path.join(GOLDEN, "over_by_hand.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            name, layers, result = (s.strip() for s in line.split("|"))
            lay = np.array([[float(x) for x in l.split()] for l in layers.split(";")])
            out.append((name, lay, np.array([float(x) for x in result.split()])))
    return out
