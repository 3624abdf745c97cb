"""The host-only units (schedule rules, samplers, selection, guided search)
built with the address and undefined-behaviour sanitizers and run over every
valid schedule of the ResNet-18 and MobileNet-v2 workloads and of a few edge
shapes, with a whole guided search over a stand-in measurement: no sanitizer
report may occur. Skipped where g++ cannot build with the sanitizers."""
import os
import subprocess

import pytest

from paper_2008_03602_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2008_03602_amd", "csrc")

EDGE_OPS = [
    W.conv("one", 1, 1, 1, 1, 1, 1, 0),                                 # a single MAC
    W.conv("dw", 2, 8, 9, 8, 3, 1, 1, groups=8),                       # depthwise, odd map
    W.Op("dil", 1, 4, 11, 11, 6, 3, 3, 1, 1, 2, 2, 2, 2, 1, 0, 0),      # dilated
    W.conv("s2", 1, 5, 13, 7, 3, 2),                                   # stride 2, odd sizes
    W.Op("gen53", 1, 4, 12, 13, 6, 5, 3, 1, 1, 2, 1, 1, 1, 1, 0, 0),    # 5x3 filter
    W.conv("tr5", 1, 6, 16, 10, 5, 1, 2),                               # rows of 16 words
]


def test_host_units_are_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "asan_host")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-pthread", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "asan_host.cpp"), os.path.join(CSRC, "schedule.cpp"),
           os.path.join(CSRC, "search.cpp"), os.path.join(CSRC, "clients.cpp"), "-o", exe]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        if "sanitize" in r.stdout or "asan" in r.stdout.lower():
            pytest.skip("g++ cannot build with the sanitizers here: " + r.stdout[-300:])
        raise AssertionError("build failed:\n" + r.stdout[-3000:])
    ops = W.config(2).ops + W.config(5).ops + EDGE_OPS
    listing = tmp_path / "ops.txt"
    listing.write_text("".join(" ".join(str(v) for v in (o.n, o.c, o.h, o.w, o.k, o.r, o.s, o.stride_h, o.stride_w,
                                                         o.pad_h, o.pad_w, o.dil_h, o.dil_w, o.groups, o.dtype,
                                                         o.layout)) + "\n" for o in ops))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    p = subprocess.run([exe, str(listing)], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env,
                       timeout=600)
    assert "Sanitizer" not in p.stdout and "runtime error" not in p.stdout, p.stdout[-4000:]
    assert p.returncode == 0, p.stdout[-4000:]
    assert "done: %d ops, 0 failures" % len(ops) in p.stdout
    # every workload op has schedules, and every op was sampled
    lines = [l for l in p.stdout.splitlines() if l.startswith("op ")]
    assert len(lines) == len(ops)
    assert all(" 0 valid" not in l for l in lines[:len(ops) - len(EDGE_OPS)])


def test_client_machinery_is_clean_under_asan_and_ubsan(tmp_path):
    # the client-thread driver of the race test, under the memory and
    # undefined-behaviour sanitizers instead
    exe = str(tmp_path / "asan_clients")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-pthread", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "tsan_clients.cpp"), os.path.join(CSRC, "clients.cpp"),
           os.path.join(CSRC, "schedule.cpp"), "-o", exe]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        if "sanitize" in r.stdout or "asan" in r.stdout.lower():
            pytest.skip("g++ cannot build with the sanitizers here: " + r.stdout[-300:])
        raise AssertionError("build failed:\n" + r.stdout[-3000:])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    p = subprocess.run([exe, str(tmp_path)], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env,
                       timeout=240)
    assert "Sanitizer" not in p.stdout and "runtime error" not in p.stdout, p.stdout[-4000:]
    assert p.returncode == 0, p.stdout[-4000:]
    assert "plain: rc 0 (expected 0)" in p.stdout
