"""The host-side ABI tests (tests/test_abi_cpu.py) once more, against a build
whose host code of the C ABI runs under AddressSanitizer and
UndefinedBehaviorSanitizer: argument checks, workspace sizing and carving
must make no out-of-bounds access, use no freed memory and hit no undefined
behaviour on the valid and the rejected calls those tests make. No GPU is
used; the sanitizer runtime is preloaded into a child interpreter (leak
checking is off: the interpreter itself keeps memory until exit)."""
import os
import subprocess
import sys

import pytest

from paper_2607_11976_amd import build as lt_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_host_code_under_asan_and_ubsan():
    rt = lt_build.sanitizer_runtime()
    if not rt:
        pytest.skip("the compiler's AddressSanitizer runtime is not installed")
    lib = lt_build.build_sanitized()
    env = dict(os.environ)
    env["LT_LIBRARY"] = lib
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = rt + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout, out[-2000:]
