"""Build the CPU oracle library (plain C, gcc, OpenMP).  Test infrastructure."""
from __future__ import annotations

import subprocess
from pathlib import Path

HERE = Path(__file__).resolve().parent
SRC = HERE / "attn_oracle.c"
LIB_PATH = HERE / "liboracle.so"

# No fast-math and no FMA contraction: the FP32 steps must round exactly as
# written.  -O2 without -march=native so the result is the same on any x86-64.
CFLAGS = ["-O2", "-std=c11", "-D_GNU_SOURCE", "-fPIC", "-shared", "-fopenmp",
          "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra", "-Wvla"]


def build() -> Path:
    tmp = LIB_PATH.with_suffix(".so.tmp")
    cmd = ["gcc", *CFLAGS, str(SRC), "-o", str(tmp), "-lm"]
    subprocess.run(cmd, check=True)
    tmp.replace(LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build())
