"""Builds libjdob.so (the C-ABI library) for gfx950 with hipcc.

Flags that matter for the results:
  -ffp-contract=off      no fused multiply-add contraction: every decision
                         follows the exact IEEE operation sequence of the ABI
  (no fast-math)         divisions stay correctly rounded
  -packed-fp32-ops off   no packed FP32 instructions are generated
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "jdob.hip")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libjdob.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def build(out: str = LIB, extra=()) -> str:
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *FLAGS, *extra, "-I", INCLUDE, "-o", tmp, SRC]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed for " + SRC)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build())
