import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


@pytest.fixture(scope="session")
def golden_dir():
    return os.path.join(ROOT, "tests", "golden")


@pytest.fixture
def launch_option():
    """Setter of library launch options (sparvar_set_launch_option) for one test;
    every option it touched is restored to its default afterwards."""
    from paper_2602_04361_amd import sparvar as sv

    touched = []

    def set_option(name, value):
        touched.append(name)
        sv.sparvar_set_launch_option(name, int(value))

    yield set_option
    for name in touched:
        sv.sparvar_set_launch_option(name, None)
