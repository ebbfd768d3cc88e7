"""The C ABI tests (tests/test_abi.py) again, against the host-sanitized build of the library
(AddressSanitizer + UndefinedBehaviorSanitizer on every host pass, device code unchanged; built by
`python -m paper_2608_27206_amd.build --sanitized` and by __graft_entry__.build()).  They exercise
argument checking, the host-only helpers, workspace sizing and the refusals that happen before any
launch, so they run on the CPU.  Any sanitizer report fails the run."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_under_address_and_undefined_behaviour_sanitizers():
    from paper_2608_27206_amd import build as b
    if not os.path.exists(b.SANITIZED_OUT):
        pytest.skip("sanitized library not built (python -m paper_2608_27206_amd.build --sanitized)")
    syms = subprocess.run(["nm", "-D", "--undefined-only", b.SANITIZED_OUT], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms, "library is not sanitized"
    rt = b.sanitizer_runtime()
    env = dict(os.environ)
    env["PACE_LIB_PATH"] = b.SANITIZED_OUT
    env["LD_PRELOAD"] = rt + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    code = ("import sys, pytest; from paper_2608_27206_amd import pace; "
            "assert pace.LIB_PATH.endswith('libpace_sanitized.so'); "
            "sys.exit(pytest.main(['-q', '-p', 'no:cacheprovider', 'tests/test_abi.py']))")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
