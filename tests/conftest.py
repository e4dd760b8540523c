import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line(
        "markers", "gpu: needs an MI355X (gfx950) GPU; runs the HIP path through the C ABI")
    config.addinivalue_line(
        "markers", "slow: full-size case (seconds to minutes)")


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    oracle._load()
    return oracle


@pytest.fixture
def knobs():
    """Set test overrides of the library (tcu_set_knob) for one test; every
    knob set is put back to 0 (the automatic choice) afterwards."""
    from paper_1908_06649_amd import tcu
    touched = []

    def put(knob: int, value: int) -> None:
        tcu.tcu_set_knob(knob, value)
        touched.append(knob)

    yield put
    for k in touched:
        tcu.tcu_set_knob(k, 0)
