"""The host-only ABI tests again, against the AddressSanitizer build of the library.

The host side of ``libmebp.so`` (argument validation, workspace layout and offsets, the
launch plans, the timing registry) is C++ that runs on every call. Here it is rebuilt with
``-fsanitize=address`` on the host pass only (device code unchanged) and the host-only
tests of ``test_abi_host.py`` run against it in a subprocess with the sanitizer runtime
preloaded: an out-of-bounds or use-after-free access in that code fails the run. Leak
checking is off: the HIP runtime keeps allocations until exit by design.

The sanitizer build takes about a minute and is reused while it is newer than every source.
"""
import glob
import os
import subprocess
import sys

import pytest

from paper_2510_03425_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _stale(lib):
    if not os.path.exists(lib):
        return True
    srcs = glob.glob(os.path.join(B.CSRC, "*")) + [os.path.join(ROOT, "include", "mebp.h"), B.__file__]
    return max(os.path.getmtime(s) for s in srcs) > os.path.getmtime(lib)


def test_host_abi_tests_pass_under_address_sanitizer():
    try:
        rt = B.asan_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = B.lib_path("asan")
    if _stale(lib):
        B.build(variant="asan")
    nm = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True)
    assert "__asan_report" in nm.stdout, "the sanitizer build carries no instrumentation"
    env = dict(os.environ, MEBP_LIB=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"),
                        "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out
