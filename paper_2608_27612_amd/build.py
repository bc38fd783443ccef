"""Builds libemr.so (the HIP library behind include/emr.h) in-tree for gfx950."""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libemr.so")
SOURCES = ["kernels.hip", "runtime.cpp", "pack.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# No packed-FP32 instructions anywhere in the device code.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def compile_cmd(out: str, extra=()):
    return ([HIPCC, "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wno-unused-function"]
            + DEVICE_FLAGS + list(extra) + [os.path.join(CSRC, s) for s in SOURCES] + ["-o", out])


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = compile_cmd(tmp)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building libemr.so")
    if verbose:
        sys.stderr.write(res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
