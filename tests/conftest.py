import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def _default_shape() -> tuple[int, int]:
    """Row-kernel shape for the whole run: CMSD_TEST_ROW_SHAPE="threads,depth" (e.g.
    "64,3") forces one for every launch of every test, so a whole suite can be run on
    each shape; unset, the library chooses per launch."""
    v = os.environ.get("CMSD_TEST_ROW_SHAPE", "")
    if not v:
        return 0, 0
    t, d = (int(x) for x in v.split(","))
    return t, d


@pytest.fixture(scope="session", autouse=True)
def _suite_row_shape():
    t, d = _default_shape()
    if (t, d) == (0, 0):
        yield
        return
    from paper_2508_15371_amd import cmsd
    cmsd.cmsd_set_row_shape(t, d)
    yield
    cmsd.cmsd_set_row_shape(0, 0)


@pytest.fixture
def row_shape():
    """set(threads, depth) forces the row kernels' workgroup size / loads in flight for
    one test (cmsd_set_row_shape; 0 keeps the per-launch choice); reset afterwards."""
    from paper_2508_15371_amd import cmsd

    def set_(threads: int = 0, depth: int = 0) -> None:
        dt, dd = _default_shape()
        cmsd.cmsd_set_row_shape(threads or dt, depth or dd)

    yield set_
    cmsd.cmsd_set_row_shape(*_default_shape())
