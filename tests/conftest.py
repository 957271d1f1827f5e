import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: long-running CPU check (opt-in through CDT_SLOW=1)")
    config.addinivalue_line("markers", "statistical: an outcome against a model's distribution "
                                       "(seeded Monte Carlo), not a parity check")


def pytest_collection_modifyitems(config, items):
    if os.environ.get("CDT_SLOW") == "1":
        return
    skip = pytest.mark.skip(reason="slow check; set CDT_SLOW=1 to run it")
    for item in items:
        if "slow" in item.keywords:
            item.add_marker(skip)


@pytest.fixture(scope="session")
def orc():
    import oracle
    oracle.lib()
    return oracle


@pytest.fixture(scope="session")
def philox_pin():
    """rocRAND's Philox4x32-10 (library routine) as a vectorised callable."""
    import ctypes

    import numpy as np

    from tests.pins import build as pins

    if not os.path.exists(pins.PHILOX_LIB):
        pins.build()
    L = ctypes.CDLL(pins.PHILOX_LIB)
    L.pin_philox4x32_10.argtypes = [ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p]
    L.pin_philox4x32_10.restype = None

    def run(ctr, key):
        ctr = np.ascontiguousarray(ctr, np.uint32).reshape(-1, 4)
        key = np.ascontiguousarray(key, np.uint32).reshape(-1, 2)
        out = np.empty_like(ctr)
        L.pin_philox4x32_10(ctr.shape[0], ctr.ctypes.data, key.ctypes.data, out.ctypes.data)
        return out

    return run
