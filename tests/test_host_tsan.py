"""The host-only client machinery (client threads, shared queue, logs, stop
and raise hooks, the watchdog) built with the thread sanitizer and run: no
data race may be reported. Skipped where g++ cannot build with
-fsanitize=thread."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2008_03602_amd", "csrc")


def test_client_machinery_is_race_free_under_tsan(tmp_path):
    exe = str(tmp_path / "tsan_clients")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=thread", "-pthread",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "tsan_clients.cpp"), os.path.join(CSRC, "clients.cpp"),
           os.path.join(CSRC, "schedule.cpp"), "-o", exe]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        if "sanitize" in r.stdout or "tsan" in r.stdout.lower():
            pytest.skip("g++ cannot build with the thread sanitizer here: " + r.stdout[-300:])
        raise AssertionError("build failed:\n" + r.stdout[-3000:])
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=66")
    p = subprocess.run([exe, str(tmp_path)], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       env=env, timeout=240)
    assert "ThreadSanitizer" not in p.stdout, p.stdout[-4000:]
    assert p.returncode == 0, p.stdout[-4000:]
    assert "plain: rc 0 (expected 0)" in p.stdout
