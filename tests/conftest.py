import json
import os
import sys
from fractions import Fraction

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def frac_matrix(rows, env=None):
    """Evaluate a fixture matrix of expression strings in exact rationals."""
    env = dict(env or {})
    ns = {"__builtins__": {}}
    ns.update(env)
    out = []
    for row in rows:
        out.append([Fraction(eval(s, ns)) if any(ch.isalpha() for ch in s) else Fraction(s) for s in row])
    return out


@pytest.fixture
def golden():
    return load_golden
