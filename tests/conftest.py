import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def load_grid_fixture(p, n):
    """Grid fixture written by tests/golden/make_grids.py (oracle only); fp64 (n, p)."""
    import numpy as np
    path = os.path.join(GOLDEN, f"grid_p{p}_n{n}.txt")
    if not os.path.exists(path):
        return None
    rows = []
    meta = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#"):
                for tok in line[1:].split():
                    if "=" in tok:
                        k, v = tok.split("=", 1)
                        meta[k] = v.rstrip(",;")
                continue
            rows.append([float(v) for v in line.split()])
    g = np.array(rows, dtype=np.float64)
    assert g.shape == (n, p), path
    return g, meta
