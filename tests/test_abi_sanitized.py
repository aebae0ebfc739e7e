"""The CPU tests of the C ABI again, against a build whose host code runs
under AddressSanitizer and UndefinedBehaviorSanitizer (validation, workspace
layout and GEMM planning of every entry point; device code is not
sanitized).  The tests run in a child process that preloads clang's ASan
runtime and loads the sanitized library through DITMI_LIB; any sanitizer
report fails the run."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    from paper_2605_25550_amd import build as B
    try:
        rt = B.sanitizer_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = B.build_sanitized(str(tmp_path_factory.mktemp("asan")))
    return lib, rt


def test_abi_suite_under_asan_ubsan(sanitized_lib):
    lib, rt = sanitized_lib
    with open(lib, "rb") as fh:
        blob = fh.read()
    assert b"__asan_report_load" in blob and b"__ubsan_handle" in blob, "host code is not instrumented"
    env = dict(os.environ, LD_PRELOAD=rt, DITMI_LIB=lib, ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    probe = ("import ctypes, os, paper_2605_25550_amd as dm; dm.lib(); "
             "assert dm.LIB_PATH == os.environ['DITMI_LIB']; "
             "assert hasattr(ctypes.CDLL(None), '__asan_init')")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_abi.py", "-q", "-x", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
