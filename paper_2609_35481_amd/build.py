"""Build the planner's HIP library for gfx950 (in-tree shared object)."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", n) for n in ("topoep.hip", "layout.hip", "gather.hip")]
SRC = SRCS[0]
LIB = os.path.join(HERE, "libtopoep.so")
INCLUDE = os.path.join(ROOT, "include")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed-FP32 instructions in any generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


# The same library with phase stamps (-DTOPOEP_STAMPS): the solver and the
# first chunk write the wall clock at phase boundaries into the workspace's
# control words.  For measurement only (bench.py --phases); the product
# library is LIB.
STAMPS_LIB = os.path.join(HERE, "libtopoep_stamps.so")


def build(verbose: bool = False) -> str:
    """Compile LIB and STAMPS_LIB (two hipcc processes side by side)."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    jobs = []
    for out, extra in ((LIB, []), (STAMPS_LIB, ["-DTOPOEP_STAMPS"])):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = [hipcc, *HIPCC_FLAGS, *extra, "-I", INCLUDE, "-o", tmp, *SRCS]
        jobs.append((out, tmp, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
    errors = []
    for out, tmp, proc in jobs:
        so, se = proc.communicate()
        if proc.returncode != 0:
            errors.append("hipcc failed for %s:\n%s%s" % (os.path.basename(out), so, se))
            continue
        if verbose:
            print(se)
        os.replace(tmp, out)
    if errors:
        raise RuntimeError("\n".join(errors))
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
