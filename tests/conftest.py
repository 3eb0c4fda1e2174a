import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: large full-size case")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_golden(name):
    """Rows of a golden fixture: '|'-separated fields, '#' starts a comment line."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([x.strip() for x in line.split("|")])
    return rows


@pytest.fixture
def golden():
    return read_golden


@pytest.fixture(params=["one_launch", "split"])
def wpath(request):
    """Runs the test once with windowed calls on the one-launch windowed
    kernel and once on the split-K + merge kernels (the library reads
    WMTP_WIN_ONE_LAUNCH_ROWS, the row threshold between them, at every call;
    0: never the one-launch kernel)."""
    key = "WMTP_WIN_ONE_LAUNCH_ROWS"
    old = os.environ.get(key)
    os.environ[key] = str(1 << 30) if request.param == "one_launch" else "0"
    yield request.param
    if old is None:
        os.environ.pop(key, None)
    else:
        os.environ[key] = old
