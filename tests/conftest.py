import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test")


@pytest.fixture(scope="session", autouse=True)
def _synth_lib():
    """Build the seeded-input generator once if it is missing."""
    from synth import gen
    if not os.path.exists(gen._LIB_PATH):
        try:
            gen.build_lib()
        except Exception:  # numpy twin is used instead
            pass
