import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def read_golden(name):
    """Parse a tests/golden/*.txt fixture: 'key: value' lines, '#' comments."""
    out = {}
    with open(os.path.join(ROOT, "tests", "golden", name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, val = line.split(":", 1)
            vals = [v.strip() for v in val.split(",")]
            out[key.strip()] = [int(v) for v in vals] if len(vals) > 1 else int(vals[0])
    return out


def same_bits(x, y) -> bool:
    """Bitwise equality of two float/complex arrays (NaN == NaN, -0 != +0)."""
    import numpy as np
    x = np.ascontiguousarray(x)
    y = np.ascontiguousarray(y)
    if x.shape != y.shape or x.dtype != y.dtype:
        return False
    w = {2: np.uint16, 4: np.uint32, 8: np.uint64, 16: np.uint64}[x.dtype.itemsize]
    return bool(np.array_equal(x.view(w), y.view(w)))
