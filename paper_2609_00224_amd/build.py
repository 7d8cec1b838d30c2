"""Build step of the HIP library: compiles csrc/*.hip for gfx950 with hipcc
into libqtea.so next to this file (in-tree, so it ships with the sources)."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", f) for f in ("qtea.hip", "grouped.hip", "grouped_mma.hip", "quant.hip")]
LIB = os.path.join(HERE, "libqtea.so")
# the debug build: unused byte values 243..255 of every decode table read NaN
LIB_DEBUG = os.path.join(HERE, "libqtea_debug.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    # keep hand-written and compiler-formed packed fp32 VALU ops out of the code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # the library's atomics are single-lane counter updates whose results are
    # used much later; the wave-level atomic rewrite would wait for every
    # outstanding load right after each of them
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
    "-Wall", "-Wno-unused-result",
]


def build(verbose: bool = False, debug: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    out = LIB_DEBUG if debug else LIB
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [hipcc, *HIPCC_FLAGS, *(["-DQTEA_DEBUG=1"] if debug else []), "-I", os.path.join(ROOT, "include"),
           "-o", tmp, *SRCS]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, debug="--debug" in sys.argv))
