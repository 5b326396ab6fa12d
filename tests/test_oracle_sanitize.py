"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/oracle_sanitize.c drives every oracle entry point on small inputs that
reach its boundary paths and checks the results against facts fixed by the
mathematics (see that file).  Here it is built together with
oracle/wf_oracle.c by gcc with -fsanitize=address,undefined (any report is
fatal) into a temporary directory and run as a child process.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_is_clean_under_sanitizers(tmp_path):
    exe = tmp_path / "oracle_sanitize"
    cmd = ["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fopenmp", "-Wall", "-Wextra",
           os.path.join(ROOT, "oracle", "wf_oracle.c"),
           os.path.join(ROOT, "tests", "oracle_sanitize.c"),
           "-o", str(exe), "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, OMP_NUM_THREADS="3",
               ASAN_OPTIONS="abort_on_error=0:halt_on_error=1:detect_leaks=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([str(exe)], capture_output=True, text=True,
                         env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "all checks hold" in res.stdout
