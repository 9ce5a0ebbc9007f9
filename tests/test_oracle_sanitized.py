"""The fp64 oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(host code only), driven by tests/oracle_sanitize_driver.c over every oracle
function on small cases with known answers (closed forms and the paper's
worked examples).  An out-of-bounds access or undefined behaviour aborts the
driver; a wrong answer makes it exit with 1."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_under_asan_and_ubsan():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "oracle_sanitized")
        cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fno-fast-math",
               "-ffp-contract=off", "-fsanitize=address,undefined",
               "-fno-sanitize-recover=all", "-Wall", "-Wextra",
               os.path.join(ROOT, "tests", "oracle_sanitize_driver.c"),
               os.path.join(ROOT, "oracle", "oracle.c"), "-lm", "-o", exe]
        build = subprocess.run(cmd, capture_output=True, text=True)
        if build.returncode != 0 and "sanitize" in build.stderr:
            pytest.skip("this gcc has no sanitizer runtime: " + build.stderr[-200:])
        assert build.returncode == 0, build.stderr
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
                   UBSAN_OPTIONS="print_stacktrace=1")
        run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
        assert run.returncode == 0, run.stdout + run.stderr
        assert "all checks passed" in run.stdout
