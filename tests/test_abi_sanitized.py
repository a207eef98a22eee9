"""The C ABI checks of test_abi_cpu.py against the host-sanitized build of the library
(AddressSanitizer + UndefinedBehaviorSanitizer on the validation, planning and launch set-up
code; built by __graft_entry__.build()), in a child process with the sanitizer runtime preloaded.
Any report aborts the child and fails the test."""
import os
import subprocess
import sys

from paper_2609_30738_amd import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_under_address_and_undefined_behaviour_sanitizers():
    assert os.path.exists(build.SAN_LIB), f"{build.SAN_LIB} missing: run __graft_entry__.build()"
    env = dict(os.environ)
    env["KVEVICT_LIB"] = build.SAN_LIB
    env["LD_PRELOAD"] = build.sanitizer_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = res.stdout[-3000:] + res.stderr[-3000:]
    assert res.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out
    assert " passed" in res.stdout
