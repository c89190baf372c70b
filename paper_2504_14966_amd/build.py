"""Builds libsloanneal.so (gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libsloanneal.so")
SRC = os.path.join(HERE, "csrc", "sloanneal.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off",
         "-fno-fast-math", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function",
         # small register arrays indexed by constants stay separate registers (split by the
         # scalar replacement pass); the target's alloca-to-vector promotion would instead
         # hold them as one vector value, copied whole wherever an element changes
         "-mllvm", "-disable-promote-alloca-to-vector"]


def build(extra: list[str] | None = None, out: str = LIB) -> str:
    tmp = out + f".tmp{os.getpid()}"
    cmd = [HIPCC, *FLAGS, *(extra or []), "-o", tmp, SRC]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(sys.argv[1:]))
