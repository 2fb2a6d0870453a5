"""The host side of the C ABI (argument validation, status codes, capacity
and workspace arithmetic, the row-stream and tile settings, the event pool's
bookkeeping) built with AddressSanitizer and UndefinedBehaviorSanitizer:
tests/test_abi_cpu.py runs against that build in a child process with the
ASan runtime preloaded, and must pass with no sanitizer report. Host only:
no kernel is launched."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc")
def test_abi_tests_pass_under_host_sanitizers():
    from paper_2510_00207_amd import build
    lib = build.build_sanitized(verbose=False)
    env = dict(os.environ)
    env.update(LD_PRELOAD=build.asan_runtime(), FLOWMOE_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"),
                        "-q", "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
    # the child really loaded the sanitized build
    probe = subprocess.run([sys.executable, "-c",
                            "import ctypes; from paper_2510_00207_amd import _lib as L; "
                            "L.load(); print(L.LIB_PATH); "
                            "print(hasattr(ctypes.CDLL(L.LIB_PATH), '__asan_report_load1'))"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert probe.returncode == 0, probe.stderr[-2000:]
    assert probe.stdout.split() == [lib, "True"], probe.stdout
