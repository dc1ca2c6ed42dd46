"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer (gcc) and run over
every exported function on small, oddly sized models (tests/oracle_sanitize.c): no
out-of-bounds access, leak or undefined arithmetic on any path the parity tests use."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_sanitize")
    src = os.path.join(ROOT, "tests", "oracle_sanitize.c")
    build = ["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", "-o", exe, src, "-lm"]
    res = subprocess.run(build, capture_output=True, text=True)
    if res.returncode != 0 and "asan" in res.stderr.lower():
        pytest.skip("this gcc has no sanitizer runtime: " + res.stderr[-200:])
    assert res.returncode == 0, res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "runtime error" not in run.stderr and "ERROR: AddressSanitizer" not in run.stderr, run.stderr
    assert "rc=0" in run.stdout
