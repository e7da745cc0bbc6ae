import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: full-size workload (seconds to minutes)")


def parse_golden(path):
    """Parse a golden fixture: '[section]' headers and 'key = v v v' lines."""
    sections, cur = {}, None
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            if line.startswith("[") and line.endswith("]"):
                cur = sections.setdefault(line[1:-1], {})
                continue
            k, v = (x.strip() for x in line.split("=", 1))
            vals = [int(x) for x in v.split()]
            cur[k] = vals[0] if len(vals) == 1 and k in ("L", "B", "H", "D", "E", "NB", "S") else vals
    return sections


def parse_pairs(path):
    """Parse 'lhs : rhs' lines of a golden fixture."""
    out = []
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                a, b = (x.strip() for x in line.split(":", 1))
                out.append((a, b))
    return out


@pytest.fixture
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")
