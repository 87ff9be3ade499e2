"""Build the gfx950 library ``libh15attn.so`` in-tree with hipcc.

Flags that matter:
  * ``-ffp-contract=off``: the H15 exponent argument must be computed by the
    fused multiply-adds written in the source and nothing else (bit-exact
    weights), and no other expression may be contracted behind our back;
  * ``-Xclang -target-feature -Xclang -packed-fp32-ops``: no packed fp32 VALU
    instructions are generated (the host pass warns that it does not know the
    feature; that is harmless).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
SRC = PKG / "csrc" / "h15attn.hip"     # kernels and their launchers
API_SRC = PKG / "csrc" / "attn_api.cpp"  # C entry points: argument checks, per-call constants
INCLUDE = ROOT / "include"
LIB_PATH = PKG / "libh15attn.so"
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-shared", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return str(Path(rocm) / "bin" / "hipcc")


# The kernel source is compiled twice: once for everything but the FP8
# lattice-weight forward kernels at d = 128, once for those alone, which are
# scheduled with the iterative ILP machine scheduler (faster for them, slower
# for the exact control and the BF16 kernels, and at d = 64 it would cost the
# third wave per SIMD).
UNITS = [
    ("kernels", SRC, []),
    ("fp8_lattice_d128", SRC, ["-DH15_FP8_LATTICE_D128=1", "-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]),
    ("api", API_SRC, []),
]


def build(extra: list[str] | None = None, verbose: bool = False) -> Path:
    import tempfile
    objdir = Path(tempfile.mkdtemp(prefix="h15attn-build-"))
    try:
        compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
        objs, procs = [], []
        for name, src, flags in UNITS:
            obj = objdir / f"{name}.o"
            cmd = [hipcc(), *compile_flags, *flags, *(extra or []), f"-I{INCLUDE}", f"-I{src.parent}", "-c",
                   str(src), "-o", str(obj)]
            procs.append((name, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
            objs.append(obj)
        failed = []
        for name, proc in procs:
            out, err = proc.communicate()
            if proc.returncode != 0:
                sys.stderr.write(out + err)
                failed.append(name)
            elif verbose:
                sys.stderr.write(err)
        if failed:
            raise RuntimeError(f"hipcc failed building {', '.join(failed)} of {LIB_PATH.name}")
        linked = objdir / LIB_PATH.name
        cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *map(str, objs), "-o", str(linked)]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc failed ({res.returncode}) linking {LIB_PATH.name}")
        check_kernel_stubs(linked)
        # the temporary folder may sit on another file system: copy next to
        # the target, then rename over it
        staged = LIB_PATH.with_name(LIB_PATH.name + ".tmp")
        shutil.copyfile(linked, staged)
        staged.chmod(0o755)
        staged.replace(LIB_PATH)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    return LIB_PATH


def check_kernel_stubs(lib: Path) -> None:
    """Refuse a library whose host side references kernel launch stubs that it
    does not define (the host compile can drop a kernel's stub without an
    error; loading the library would then fail)."""
    res = subprocess.run(["nm", "-D", "--undefined-only", str(lib)], capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"nm failed on {lib.name}: {res.stderr.strip()}")
    missing = [ln.split()[-1] for ln in res.stdout.splitlines() if "__device_stub__" in ln]
    if missing:
        lib.unlink(missing_ok=True)
        raise RuntimeError(f"{lib.name}: {len(missing)} kernel launch stubs are undefined, e.g. {missing[0]}")


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
