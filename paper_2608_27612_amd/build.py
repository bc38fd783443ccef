"""Builds libemr.so (the HIP library behind include/emr.h) in-tree for gfx950: first the template
code object of the compiled tier (jit.hip -> libemr_jit.co), which the library embeds, then the
library itself."""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libemr.so")
JIT_CO = os.path.join(HERE, "libemr_jit.co")
SOURCES = ["kernels.hip", "phase2.hip", "runtime.cpp", "pack.cpp", "plan.cpp", "sched.cpp",
           "jit.cpp", "jit_image.cpp", "record_file.cpp", "network.hip", "net_sort.hip", "band.hip",
           "networks.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# No packed-FP32 instructions anywhere in the device code. Atomics stay as written: in the discover
# path every atomic on one address is issued by a single lane, so the compiler's rewrite of
# wave-wide atomics (a loop over the active lanes) would only add code.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]


def template_cmd(out: str):
    return ([HIPCC, "-O3", "-std=c++17", "-Wall", "--genco", "--cuda-device-only",
             "--no-gpu-bundle-output"] + DEVICE_FLAGS + [os.path.join(CSRC, "jit.hip"), "-o", out])


def compile_cmd(out: str, extra=()):
    return ([HIPCC, "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall", "-Wno-unused-function",
             '-DEMR_JIT_TEMPLATE="%s"' % JIT_CO]
            + DEVICE_FLAGS + list(extra) + [os.path.join(CSRC, s) for s in SOURCES] + ["-o", out])


def _run(cmd, what):
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("hipcc failed building " + what)
    return res


def build(verbose: bool = False) -> str:
    tmp = JIT_CO + ".tmp%d" % os.getpid()
    _run(template_cmd(tmp), "libemr_jit.co")
    os.replace(tmp, JIT_CO)
    tmp = LIB + ".tmp%d" % os.getpid()
    res = _run(compile_cmd(tmp), "libemr.so")
    if verbose:
        sys.stderr.write(res.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
