"""The C-ABI tests of test_abi_cpu.py against a host-sanitized build of the library (CPU only).

build.build_sanitized() compiles api.cpp (argument validation, workspace layout and
sizing, launch set-up) with AddressSanitizer and UndefinedBehaviorSanitizer; the
tests then run in a child interpreter with the sanitizer runtimes preloaded, so an
out-of-bounds access, use after free, signed overflow or misaligned access on the
host side of any call aborts the run.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(os.environ.get("TGVKV_LIBRARY") is not None, reason="already running against another build")
def test_abi_tests_pass_under_asan_and_ubsan():
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("gcc sanitizer runtimes not installed")
    sys.path.insert(0, ROOT)
    from paper_2606_03075_amd import build
    lib = build.build_sanitized()
    env = dict(os.environ)
    env["TGVKV_LIBRARY"] = lib
    env["LD_PRELOAD"] = ":".join(p for p in (asan, ubsan, env.get("LD_PRELOAD")) if p)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["CUDA_VISIBLE_DEVICES"] = ""
    env["HIP_VISIBLE_DEVICES"] = ""
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
