"""The host-only C ABI checks (tests/test_abi.py) rerun against a build of the
library whose host code (argument validation, geometry tables) is instrumented
with AddressSanitizer and UndefinedBehaviorSanitizer; any report fails the run.
CPU only: no call in those tests reaches a kernel launch."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_under_asan_and_ubsan():
    from paper_2602_04361_amd import build_host_sanitized as bhs

    if not os.path.exists(os.path.join(bhs.BUILD, "api.o")):
        pytest.skip("library objects not built (python -m paper_2602_04361_amd.build)")
    lib = bhs.build()
    asan = bhs.asan_runtime()
    assert os.path.isabs(asan) and os.path.exists(asan), asan
    env = dict(os.environ, LD_PRELOAD=asan, SPARVAR_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # the sanitized library is the one loaded, with the ASan runtime in the process
    probe = ("from paper_2602_04361_amd import sparvar as sv; sv.load_library(); "
             "m = open('/proc/self/maps').read(); "
             "assert 'libsparvar_host_sanitized.so' in m and 'libasan' in m and 'libsparvar.so' not in m")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join("tests", "test_abi.py")], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
