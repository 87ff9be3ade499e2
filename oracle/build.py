"""Build the CPU oracle library (plain C, gcc, OpenMP).  Test infrastructure."""
from __future__ import annotations

import subprocess
import sys
from pathlib import Path

HERE = Path(__file__).resolve().parent
SRC = HERE / "attn_oracle.c"
LIB_PATH = HERE / "liboracle.so"

# No fast-math and no FMA contraction: the FP32 steps must round exactly as
# written.  -O2 without -march=native so the result is the same on any x86-64.
CFLAGS = ["-O2", "-std=c11", "-D_GNU_SOURCE", "-fPIC", "-shared", "-fopenmp",
          "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra", "-Wvla"]
# AddressSanitizer and UndefinedBehaviorSanitizer build (every report fatal);
# the process that loads it must preload gcc's libasan (sanitizer_preload()).
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all"]


def build(dest: Path | None = None, sanitize: bool = False) -> Path:
    out = Path(dest) if dest is not None else LIB_PATH
    tmp = out.with_suffix(".so.tmp")
    cmd = ["gcc", *CFLAGS, *(SANITIZE_FLAGS if sanitize else []), str(SRC), "-o", str(tmp), "-lm"]
    subprocess.run(cmd, check=True)
    tmp.replace(out)
    return out


def sanitizer_preload() -> str:
    """Path of gcc's AddressSanitizer runtime, for LD_PRELOAD."""
    res = subprocess.run(["gcc", "-print-file-name=libasan.so"], check=True, capture_output=True, text=True)
    return res.stdout.strip()


if __name__ == "__main__":
    print(build(sanitize="--sanitize" in sys.argv))
