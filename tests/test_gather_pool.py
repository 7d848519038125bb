"""The staged fetch path's host worker pool (paper_2608_07009_amd/csrc/gather_pool.h), built on
its own with ThreadSanitizer (host code, g++): every index of every job handed out exactly
once, in whole grains, with no data race reported."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_gather_pool_under_thread_sanitizer(tmp_path):
    exe = str(tmp_path / "gather_pool_check")
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=thread", "-pthread",
                           "-I", os.path.join(ROOT, "paper_2608_07009_amd", "csrc"),
                           os.path.join(ROOT, "tests", "gather_pool_check.cc"), "-o", exe])
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=66")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr[-3000:]
    assert r.stdout.startswith("ok"), r.stdout
    assert "WARNING: ThreadSanitizer" not in r.stderr, r.stderr[-3000:]
