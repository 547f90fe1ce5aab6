import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")


GOLDEN = os.path.join(ROOT, "tests", "golden")


def paper_values():
    """Parse tests/golden/paper_values.txt into {key: [ints]}."""
    out = {}
    with open(os.path.join(GOLDEN, "paper_values.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, vals, _cite = [x.strip() for x in line.split("|")]
            out[key] = [int(v) for v in vals.split()]
    return out


@pytest.fixture(scope="session")
def paper():
    return paper_values()
