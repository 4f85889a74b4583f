"""The C ABI's host-side validation under AddressSanitizer and UBSan (no GPU).

The library is built with both sanitizers on its host code (the device code
as usual), and the ABI contract tests of test_abi.py run against it in a
child process with the sanitizer runtime preloaded: any sanitizer report ends
the child with an error.  Every call those tests make is refused on the host
before device work, so nothing here launches a kernel.
"""
import os
import subprocess
import sys

import pytest

from paper_2211_12858_amd import build as sb_build

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def test_abi_contract_under_host_sanitizers(tmp_path):
    try:
        sb_build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc is not available")
    rt = sb_build.sanitizer_runtime()
    if rt is None:
        pytest.skip("the clang AddressSanitizer runtime is not available")
    lib = str(tmp_path / "libsketchboost_san.so")
    sb_build.build_host_sanitized(lib)
    undefined = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in undefined and "__ubsan_handle" in undefined, "the build is not instrumented"
    env = dict(os.environ, LD_PRELOAD=rt, SKETCHBOOST_LIB=lib,
               # the HIP runtime's own allocations at exit are not this library's leaks
               ASAN_OPTIONS="detect_leaks=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                          os.path.join(HERE, "test_abi.py")], env=env, cwd=ROOT, capture_output=True, text=True,
                         timeout=900)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in res.stdout
