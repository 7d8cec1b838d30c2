"""Host checks of the planner, the packed layout's regions and the chunk
queue protocol (tests/host/plan_check.cpp), compiled from the library's own
host headers with the address and undefined-behaviour sanitizers and run on
the CPU.  The program's header lists what it checks; among them, that every
problem record's pointers (the vs words included) are its matrix's base plus
the region offsets, each region inside bytes_total."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "plan_check.cpp")
INCLUDES = [os.path.join(ROOT, "include"), os.path.join(ROOT, "paper_2609_00224_amd", "csrc")]


def _build(tmp_path, sanitize=True):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "plan_check")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror"]
    if sanitize:
        cmd += ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    for inc in INCLUDES:
        cmd += ["-I", inc]
    cmd += ["-o", exe, SRC]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def test_plan_records_layout_and_queue_under_sanitizers(tmp_path):
    exe = _build(tmp_path)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    for group in ("layout regions", "plan records", "planner argument checks", "chunk queue model",
                  "one-matrix runs"):
        assert f"ok {group}" in r.stdout, r.stdout
