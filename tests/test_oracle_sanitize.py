"""The oracle built with the address and undefined-behaviour sanitizers
(gcc -fsanitize=address,undefined, no recovery) and run by a driver that
calls every oracle function on small random and edge-case inputs: no
out-of-bounds access, leak or undefined operation in the oracle."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "oracle_sanitize")
        cmd = ["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-pthread",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
               "-I", os.path.join(ROOT, "oracle"), os.path.join(ROOT, "oracle", "oracle.c"),
               os.path.join(ROOT, "tests", "oracle_sanitize_main.c"), "-o", exe, "-lm"]
        subprocess.run(cmd, check=True, capture_output=True, text=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
        for threads in ("1", "4"):  # plain loops, then items spread over threads
            r = subprocess.run([exe, threads], capture_output=True, text=True, env=env, timeout=600)
            assert r.returncode == 0, r.stdout + r.stderr
            assert "ok" in r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_threads_under_thread_sanitizer():
    """The same driver with the oracle's items spread over 4 threads, built
    with ThreadSanitizer: a data race between two items aborts the run."""
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "oracle_tsan")
        cmd = ["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-pthread",
               "-fsanitize=thread", "-I", os.path.join(ROOT, "oracle"), os.path.join(ROOT, "oracle", "oracle.c"),
               os.path.join(ROOT, "tests", "oracle_sanitize_main.c"), "-o", exe, "-lm"]
        subprocess.run(cmd, check=True, capture_output=True, text=True)
        env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1:exitcode=66")
        r = subprocess.run([exe, "4"], capture_output=True, text=True, env=env, timeout=600)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "ok" in r.stdout
