"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The C-ABI front end (``api.cpp``: argument validation, stride and overlap
checks, workspace sizing, dispatch) is built for the host with both
sanitizers, its kernel launchers replaced by stand-ins that report that no
device is present (``tests/sanitize/launch_stub.cpp``); the oracle is built
the same way.  The CPU tests of the API and of the oracle then run in a child
process against those builds, with the ASan runtime preloaded and every
sanitizer report fatal.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_07713_amd", "csrc")
SAN_FLAGS = ["-O1", "-g", "-fPIC", "-shared", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"


@pytest.fixture(scope="module")
def sanitized_libs(tmp_path_factory):
    if not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("HIP headers not installed")
    d = tmp_path_factory.mktemp("san")
    api = str(d / "libmoa_attn_san.so")
    _run(["g++", "-std=c++17", *SAN_FLAGS, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
          os.path.join(CSRC, "api.cpp"), os.path.join(ROOT, "tests", "sanitize", "launch_stub.cpp"),
          "-o", api, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"])
    orc = str(d / "liboracle_attn_san.so")
    _run(["gcc", "-std=c11", *SAN_FLAGS, "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          os.path.join(ROOT, "oracle", "oracle_attn.c"), "-o", orc, "-lm"])
    for lib in (api, orc):
        syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
        assert "__asan_" in syms and "__ubsan_handle_" in syms, f"{lib} is not instrumented"
    return api, orc


def test_api_and_oracle_tests_under_sanitizers(sanitized_libs):
    if not os.path.exists(os.path.join(ROOT, "paper_2606_07713_amd", "libmoa_attn.so")):
        pytest.skip("HIP library not built (the binding needs it to import)")
    api, orc = sanitized_libs
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    env = dict(os.environ)
    env.update(LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               MOA_TEST_SANITIZED_API_LIB=api, MOA_TEST_SANITIZED_ORACLE_LIB=orc,
               OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", "tests/test_api.py", "tests/test_oracle.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    tail = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr and "runtime error:" not in r.stderr, tail
    assert " passed" in r.stdout and " skipped" not in r.stdout.split("\n")[-2], tail
