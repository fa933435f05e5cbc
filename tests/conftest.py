import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionfinish(session, exitstatus):
    """With the uniformity-checking build loaded (RKC_LIBRARY=.../librkc_check.so), fail the session
    when any kernel's readfirstlane saw active lanes that disagreed."""
    mod = sys.modules.get("paper_2605_24259_amd")
    lib = getattr(mod, "_lib", None) if mod else None
    if lib is None or not hasattr(lib, "rkc_debug_uniform_violations"):
        return
    lib.rkc_debug_uniform_violations.restype = __import__("ctypes").c_uint32
    n = int(lib.rkc_debug_uniform_violations())
    print(f"\nuniformity check: {n} readfirstlane calls with disagreeing lanes", flush=True)
    if n:
        session.exitstatus = 1


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    return oracle


@pytest.fixture(scope="session")
def tg():
    from paper_2605_24259_amd import tracegen
    return tracegen
