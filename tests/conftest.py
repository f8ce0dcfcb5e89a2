import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU test")


GOLDEN = os.path.join(ROOT, "tests", "golden")


def read_golden(name):
    """Parse a golden text fixture: '# comment' lines are skipped; other lines are
    'key v1 v2 ...'. 'req' lines are collected in order."""
    out = {"req": []}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            if key == "req":
                i = vals.index("live")
                j = vals.index("table")
                out["req"].append(dict(live=[int(x) for x in vals[i + 1:j]],
                                       table=[int(x) for x in vals[j + 1:]]))
            else:
                out[key] = vals
    return out
