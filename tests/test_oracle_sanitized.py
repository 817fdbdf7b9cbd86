"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer (gcc, on the CPU): the
oracle's own test files run against that build in a child process, and any sanitizer report
(an out-of-bounds access, a float-to-integer conversion out of range, a signed overflow, a bad
shift) fails the run."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TESTS = ["tests/test_oracle_coder.py", "tests/test_oracle_fit.py",
         "tests/test_oracle_quantizer.py", "tests/test_oracle_codec.py",
         "tests/test_oracle_tokens.py"]


def _asan_runtime():
    out = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.timeout(900)
def test_oracle_tests_pass_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_asan.so"))
    env = dict(os.environ)
    env.update({
        "CG_ORACLE_LIB": lib,
        "LD_PRELOAD": rt,
        # leaks of the interpreter itself are not the oracle's; stop at the first report
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1:exitcode=77",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1:exitcode=78",
    })
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu and not slow",
           "-p", "no:cacheprovider", *TESTS]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=880)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, tail
