"""The host ABI tests once more, against the argument-validation layer built with
g++ under AddressSanitizer and UndefinedBehaviorSanitizer.

api.cpp (every entry point's validation, the workspace sizes, the per-thread error
message) includes no HIP header, so it builds with the host compiler alone; linked
with host stand-ins for the launchers it gives a GPU-free library with the same
exports. tests/test_abi_host.py runs against it in a child process that preloads
the sanitizer runtimes; any report fails the run.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def _runtime(name):
    r = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(600)
def test_abi_host_under_sanitizers():
    from paper_2607_07508_amd import build as B
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if asan is None or ubsan is None:
        pytest.skip("g++ sanitizer runtimes not installed")
    lib = B.build_host_check(sanitize=True)
    env = dict(os.environ)
    env["LD_PRELOAD"] = f"{asan}:{ubsan}"
    # leak checking would report the interpreter's own allocations at exit
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:exitcode=86"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1:exitcode=87"
    code = ("import sys, pytest\n"
            "from paper_2607_07508_amd import binding\n"
            "binding.LIB_PATH = sys.argv[1]\n"
            "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', 'tests/test_abi_host.py']))\n")
    r = subprocess.run([sys.executable, "-c", code, lib], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=540)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
