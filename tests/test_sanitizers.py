"""CPU sanitizer builds, AddressSanitizer and UndefinedBehaviorSanitizer with
every report fatal:
  * the oracle library (oracle/attn_oracle.c);
  * the host side of the GPU library: the C entry points with their argument
    checks, per-call constants, decode cut and workspace sizing
    (csrc/attn_api.cpp), built with a host compiler alone and linked with
    launchers that launch nothing (tests/sanitize_launch_stub.cpp).
A child process with gcc's ASan runtime preloaded then runs the oracle tests
(all but the three exhaustive fp32 sweeps, which only loop over arithmetic)
and the ABI tests against these builds (H15_ORACLE_LIB, H15ATTN_LIB)."""
import os
import subprocess
import sys
from pathlib import Path

import pytest

from oracle import build as obuild

ROOT = Path(__file__).resolve().parent.parent
CSRC = ROOT / "paper_2609_33586_amd" / "csrc"
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
TESTS = ["tests/test_abi.py", "tests/test_oracle_h15.py", "tests/test_oracle_attn.py", "tests/test_oracle_sq.py",
         "tests/test_oracle_tau.py", "tests/test_oracle_decode.py", "tests/test_lane_recipe.py",
         "tests/test_lse_bound.py"]

CHECK_LOADED = """
import ctypes, oracle, paper_2609_33586_amd as pkg
assert hasattr(ctypes.CDLL(None), '__asan_init'), 'ASan runtime not loaded'
assert oracle.lib()._name == {olib!r}, oracle.lib()._name
L = pkg.lib()
assert L._name == {hlib!r} and L.h15_stub_launches() == 0
print('sanitized builds loaded')
"""


@pytest.fixture(scope="module")
def builds(tmp_path_factory):
    d = tmp_path_factory.mktemp("sanitize")
    olib = obuild.build(d / "liboracle_san.so", sanitize=True)
    hlib = d / "libh15attn_host_san.so"
    subprocess.run(["g++", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off", "-Wall", "-Wextra", "-Werror", *SAN,
                    f"-I{ROOT / 'include'}", f"-I{CSRC}", str(CSRC / "attn_api.cpp"),
                    str(ROOT / "tests" / "sanitize_launch_stub.cpp"), "-o", str(hlib)], check=True)
    env = dict(os.environ, LD_PRELOAD=obuild.sanitizer_preload(), ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", H15_ORACLE_LIB=str(olib), H15ATTN_LIB=str(hlib))
    return olib, hlib, env


def run(cmd, env):
    res = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout + res.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert res.returncode == 0, out[-4000:]
    return out


def test_sanitized_builds_load(builds):
    olib, hlib, env = builds
    out = run([sys.executable, "-c", CHECK_LOADED.format(olib=str(olib), hlib=str(hlib))], env)
    assert "sanitized builds loaded" in out


def test_oracle_and_abi_tests_under_sanitizers(builds):
    _, _, env = builds
    out = run([sys.executable, "-m", "pytest", *TESTS, "-q", "-p", "no:cacheprovider", "-k", "not exhaustive"], env)
    assert " passed" in out and " failed" not in out and " error" not in out, out[-2000:]
