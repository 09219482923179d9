import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs a real MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "sanitize: builds the host code with ASan/UBSan and reruns host tests")
    _use_sanitized_builds()


def _use_sanitized_builds():
    """Under tests/test_host_sanitizers.py the host tests run in a child
    process against sanitized builds: ROCKET_TEST_HOST_LIB names a host-only
    build of the generator, planner tables and MINIROCKET fit, and
    ROCKET_TEST_ORACLE_LIB a build of the oracle's C library (both with
    AddressSanitizer and UndefinedBehaviorSanitizer)."""
    host = os.environ.get("ROCKET_TEST_HOST_LIB")
    if host:
        import ctypes
        from paper_2601_17091_amd import rocket as rb
        rb.LIB_PATH = host
        rb._lib = rb.bind(ctypes.CDLL(host), rb.HOST_SYMBOLS)
    orc = os.environ.get("ROCKET_TEST_ORACLE_LIB")
    if orc:
        from oracle import rocket_oracle
        rocket_oracle._LIB_PATH = orc
        rocket_oracle._lib = None
    if host or orc:
        print("[sanitized builds] host=%s oracle=%s" % (host, orc), flush=True)


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.fixture(scope="session")
def oracle():
    from oracle import rocket_oracle
    rocket_oracle.build()
    return rocket_oracle
