"""The oracle under the host sanitizers: oracle.c and a C driver
(tests/oracle_sanitize.c) that calls every entry point of oracle.h on seeded
random heterographs are built with gcc, AddressSanitizer and
UndefinedBehaviorSanitizer, and run; any sanitizer report, leak or wrong
status fails the test.  CPU only."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ORACLE = os.path.join(ROOT, "oracle")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_sanitize")
    build = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
             "-Wall", "-Wextra", "-Wno-unknown-pragmas", "-I", ORACLE,
             os.path.join(ORACLE, "oracle.c"), os.path.join(HERE, "oracle_sanitize.c"),
             "-o", exe]
    res = subprocess.run(build, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe, "60"], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-4000:]
    assert "runtime error" not in run.stderr, run.stderr[-4000:]
    assert "every call as expected" in run.stdout
