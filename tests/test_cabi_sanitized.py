"""tests/test_cabi.py again, against the library whose host code (argument
checks, workspace sizing, plan checks, error reporting) is built with
AddressSanitizer and UndefinedBehaviorSanitizer, in a child process with the
sanitizer runtime preloaded. Any report ends the child with an error."""

import os
import subprocess
import sys

import pytest

from paper_2607_01308_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = [os.path.join(build.CSRC, "api.cpp"), os.path.join(build.CSRC, "internal.h"),
           os.path.join(ROOT, "include", "cmerge.h")]

CHILD = """
import ctypes, sys
sys.path.insert(0, sys.argv[3])
import paper_2607_01308_amd._cabi as C
C.LIB_PATH = sys.argv[1]
assert C.lib()._name == sys.argv[1]
assert hasattr(ctypes.CDLL(None), "__asan_init"), "sanitizer runtime not loaded"
import pytest
sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", sys.argv[2]]))
"""


@pytest.mark.skipif(bool(os.environ.get("LD_PRELOAD")),
                    reason="this process already preloads a library; the sanitizer runtime "
                           "must come first")
def test_cabi_under_address_and_undefined_behavior_sanitizers():
    lib = build.SAN_LIB
    if not os.path.exists(lib) or os.path.getmtime(lib) < max(os.path.getmtime(s) for s in SOURCES):
        build.build_sanitized()
    env = dict(os.environ, LD_PRELOAD=build.sanitizer_runtime(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", CHILD, lib, os.path.join(ROOT, "tests", "test_cabi.py"),
                        ROOT], env=env, capture_output=True, text=True, timeout=600, cwd=ROOT)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, out
    assert " passed" in r.stdout, out
