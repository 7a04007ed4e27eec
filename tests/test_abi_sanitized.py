"""The host side of the C ABI (configuration checks, buffer layout, context
handling, argument validation) under AddressSanitizer and
UndefinedBehaviorSanitizer: the host code of dms_api.hip is rebuilt with
both (build.build_sanitized) and tests/test_abi.py runs against that library
in a subprocess with the sanitizer runtime preloaded.  Any report fails the
run (halt_on_error).  CPU only: no kernel is launched."""
import os
import subprocess
import sys

from paper_2506_05345_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_under_address_and_undefined_behaviour_sanitizers():
    lib = build.build_sanitized()
    # the library is instrumented: it calls into both sanitizer runtimes
    syms = subprocess.run(["nm", "-D", lib], stdout=subprocess.PIPE, text=True, check=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms
    env = dict(os.environ)
    env.update(LD_PRELOAD=build.sanitizer_runtime(), DMS_TEST_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"),
                        "-q", "-m", "not gpu", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=600)
    out = r.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out, out[-2000:]
