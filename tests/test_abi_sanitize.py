"""The C ABI's host code under AddressSanitizer and UBSan (CPU only): a
sanitized build of the library linked with tests/abi_check.cpp, which calls
the ranking entry point on random and tied scores and every entry point's
argument validation.  Any sanitizer report fails the test."""
import os
import subprocess

from paper_2607_23159_amd import build


def test_abi_under_address_and_undefined_behaviour_sanitizers():
    exe = build.build_abi_check()
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ABI CHECK OK" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
