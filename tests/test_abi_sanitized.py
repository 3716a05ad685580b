"""The argument-validation cases of tests/test_abi.py against a build of the
C-ABI glue under AddressSanitizer and UBSan (host code, gcc; no GPU needed):
every check must pass with no sanitizer report."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++ with the ASan/UBSan runtimes")
def test_validation_under_sanitizers():
    from paper_2606_05742_amd import build
    lib = build.build_host_sanitized()
    env = dict(os.environ, ADAPLD_LIB=lib, LD_PRELOAD=build.sanitizer_preload(),
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # the child loads the sanitized build, with the sanitizer runtimes live
    probe = ("import ctypes, sys; ctypes.CDLL(None).__asan_report_load4; "
             "from paper_2606_05742_amd import binding; "
             "assert binding.LIB_PATH == sys.argv[1], binding.LIB_PATH; binding.load_library(); print('ok')")
    r = subprocess.run([sys.executable, "-c", probe, lib], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "tests/test_abi.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert "passed" in out
