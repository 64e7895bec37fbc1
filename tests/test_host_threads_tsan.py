"""ThreadSanitizer on the host concurrency (CPU only): the CPU share's worker team and
the pin team, built with g++ -fsanitize=thread into a stand-alone driver
(tests/tsan/host_threads_check.cpp) and run; any race report or wrong result fails."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2403_01164_amd", "csrc")


def test_worker_team_and_pin_team_under_thread_sanitizer(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "host_threads_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=thread", "-fopenmp",
           os.path.join(CSRC, "cpu_share.cpp"), os.path.join(ROOT, "tests", "tsan", "host_threads_check.cpp"),
           "-o", exe, "-lpthread"]
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert b.returncode == 0, b.stderr[-3000:]
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=66 second_deadlock_stack=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert "ThreadSanitizer" not in r.stderr, r.stderr[-6000:]
    assert r.returncode == 0 and "host thread check ok" in r.stdout, (r.returncode, r.stdout, r.stderr[-3000:])
