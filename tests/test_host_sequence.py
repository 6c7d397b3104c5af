"""The reservoir's host call protocol under the thread sanitizer (CPU only).

Builds tests/host/reservoir_sequence.cpp against the library's own
res_host.h with g++ -fsanitize=thread and runs it: concurrent puts and draws
must be ordered by consecutive tickets, replay in ticket order must reproduce
every call's kernel arguments, and the sanitizer must report nothing.  A
second build plants an unlocked read, which the sanitizer must report.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "host", "reservoir_sequence.cpp")
INC = [os.path.join(ROOT, "include"), os.path.join(ROOT, "paper_2309_16743_amd", "csrc")]


def _build(tmp_path, extra=()):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = os.path.join(str(tmp_path), "seq" + ("_race" if extra else ""))
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=thread", *[f"-I{d}" for d in INC], *extra, SRC, "-o", exe,
           "-pthread"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return exe


def _run(exe):
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1 exitcode=66")
    return subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)


def test_concurrent_calls_follow_ticket_order_without_races(tmp_path):
    res = _run(_build(tmp_path))
    assert "ThreadSanitizer" not in res.stderr, res.stderr[-4000:]
    assert res.returncode == 0, res.stdout + res.stderr[-2000:]
    assert res.stdout.strip().endswith("ok")
    for policy in (0, 1, 2):
        assert f"policy {policy}:" in res.stdout


def test_planted_unlocked_read_is_reported(tmp_path):
    res = _run(_build(tmp_path, ("-DPLANT_RACE",)))
    assert res.returncode == 66 and "data race" in res.stderr, res.stderr[-2000:]
