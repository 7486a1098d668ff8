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


# Sanitizer runs (tests/test_sanitizers.py start pytest in a child process with
# these variables set): the C-ABI front end and the oracle built with
# AddressSanitizer and UndefinedBehaviorSanitizer stand in for the normal
# builds, so the CPU tests of both exercise the instrumented host code.
_SAN_API = os.environ.get("MOA_TEST_SANITIZED_API_LIB")
_SAN_ORACLE = os.environ.get("MOA_TEST_SANITIZED_ORACLE_LIB")
if _SAN_API:
    import ctypes

    _REAL_API = os.path.join(ROOT, "paper_2606_07713_amd", "libmoa_attn.so")
    _CDLL = ctypes.CDLL

    class _RedirectCDLL(_CDLL):
        def __init__(self, name, *args, **kwargs):
            if name and os.path.abspath(name) == _REAL_API:
                name = _SAN_API
            super().__init__(name, *args, **kwargs)

    ctypes.CDLL = _RedirectCDLL
if _SAN_ORACLE:
    import oracle

    oracle._LIB_PATH = _SAN_ORACLE
