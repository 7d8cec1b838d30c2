"""The oracle's and the generator's C code under the host address and
undefined-behaviour sanitizers: both libraries are rebuilt with
-fsanitize=address,undefined and the oracle, quantizer-oracle and generator
CPU tests run again against those builds, in a child process with the
sanitizer runtime preloaded (the Python interpreter is not built with it).
Any out-of-bounds access, use after free or undefined arithmetic in the C
code ends the child with the sanitizer's report."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no gcc")
    path = subprocess.run([gcc, f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip(f"{name} not found")
    return path


def test_oracle_and_generator_tests_under_sanitizers(tmp_path):
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    env = dict(os.environ)
    env.update(
        QTEA_ORACLE_LIB=oracle.build_sanitized(str(tmp_path)),
        QTEA_SYNTH_LIB=synth.build_sanitized(str(tmp_path)),
        LD_PRELOAD=f"{asan}:{ubsan}",
        # CPython's own allocations are not freed at exit: leaks are not
        # checked; every other report ends the process with status 1
        ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
        UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
        OMP_NUM_THREADS="4",
    )
    tests = [os.path.join(ROOT, "tests", t) for t in ("test_oracle.py", "test_synth.py", "test_quant_oracle.py")]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider", *tests],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-4000:] + r.stderr[-4000:])
    assert " passed" in r.stdout
