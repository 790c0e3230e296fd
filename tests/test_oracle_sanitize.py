"""Sanitizer build of the CPU oracle (host code only).

oracle/oracle.c is compiled together with tests/oracle_sanitize_main.c under AddressSanitizer
and UndefinedBehaviorSanitizer, and the driver calls every oracle entry point on small
seeded inputs and edge cases (empty batches, K = 1 and K = N, tied and -inf logits, NULL
optional outputs, invalid arguments, bad expert ids).  The run must end cleanly: an
out-of-bounds access, a use after free or undefined behaviour in the oracle aborts it.
Built without OpenMP, so that the sanitizers see one thread.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_address_and_ub_sanitizers():
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "oracle_sanitized")
        cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
               "-Wall", "-Wno-unknown-pragmas",
               os.path.join(ROOT, "oracle", "oracle.c"),
               os.path.join(HERE, "oracle_sanitize_main.c"), "-lm", "-o", exe]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        if r.returncode != 0 and "sanitize" in r.stdout and "cannot find" in r.stdout:
            pytest.skip("sanitizer runtime not installed: " + r.stdout[-300:])
        assert r.returncode == 0, r.stdout
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1")
        run = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                             env=env, timeout=120)
        assert run.returncode == 0, run.stderr[-4000:]
        assert "runtime error" not in run.stderr, run.stderr[-4000:]
        assert "oracle sanitizer run: ok" in run.stdout
