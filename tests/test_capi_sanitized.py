"""The host runtime's argument checks under AddressSanitizer and UndefinedBehaviorSanitizer.

api.cpp (validation, planning, the C ABI) is built with both sanitizers for the host pass only
and -fno-sanitize-recover, linked with the ordinary kernel objects, and the C-ABI CPU tests run
again against it in a child process that preloads the sanitizer runtime.  No GPU is needed: no
call in those tests reaches a kernel."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc_present() -> bool:
    return bool(os.environ.get("HIPCC") or os.path.exists("/opt/rocm/bin/hipcc") or shutil.which("hipcc"))


@pytest.mark.skipif(not _hipcc_present(), reason="hipcc not available")
def test_capi_checks_clean_under_asan_and_ubsan():
    from paper_2608_08340_amd import build

    lib = build.build_sanitized()
    rt = build.asan_runtime()
    nm = shutil.which("nm")
    if nm:  # the host code is instrumented
        und = subprocess.run([nm, "-D", "--undefined-only", lib], capture_output=True, text=True).stdout
        assert "__asan_" in und and "__ubsan_handle_" in und
    env = dict(os.environ, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    code = ("import sys, pytest\n"
            "import paper_2608_08340_amd as P\n"
            f"P.LIB_PATH = {lib!r}\n"
            "P._lib = None\n"
            f"sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', {os.path.join(ROOT, 'tests', 'test_capi_cpu.py')!r}]))\n")
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=600, cwd=ROOT)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert " passed" in r.stdout and "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out
