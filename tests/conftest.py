import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: full-size workloads (minutes of CPU oracle time)")


@pytest.fixture
def tune():
    """``tune(name, value)`` sets one of the library's test settings
    (``ssd_set_tuning``); every setting made is put back to 0 afterwards."""
    from paper_2405_21060_amd import ssd

    names = []

    def set_(name, value):
        rc = ssd.ssd_set_tuning(name, int(value))
        assert rc == ssd.SSD_OK, (name, value, rc)
        names.append(name)

    yield set_
    for n in names:
        ssd.ssd_set_tuning(n, 0)
