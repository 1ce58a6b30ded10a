import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built libesb.so")


def read_golden(name):
    """Rows of whitespace-separated fields from tests/golden/<name>, '#' starts a comment."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


# (b, k_sig) pairs of the paper's Table 1 (paper k = k_sig - 1).
TABLE1_BK = [(2, 1), (3, 1), (3, 2), (4, 1), (4, 2), (4, 3), (5, 2), (5, 3), (5, 4),
             (6, 3), (6, 4), (6, 5), (7, 4), (7, 5), (7, 6), (8, 5), (8, 6), (8, 7)]
ALL_BK = [(b, ks) for b in range(2, 9) for ks in range(1, b)]
