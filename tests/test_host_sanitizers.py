"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer:
the library's host sources (argument validation, tree mask and sparse-tree
builders, workspace layout) are rebuilt with both sanitizers, and the
host-only ABI tests run against that build in a child process with the
sanitizer runtime preloaded.  Any out-of-bounds access, use after free or
undefined behaviour aborts the child."""
import os
import subprocess
import sys

from paper_2405_18628_amd.build import build_host_sanitized, sanitizer_runtime

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_host_code_clean_under_asan_and_ubsan():
    lib = build_host_sanitized()
    env = dict(os.environ, LD_PRELOAD=sanitizer_runtime(), PPD_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout
