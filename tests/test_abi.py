"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects invalid arguments before touching the GPU."""
import ctypes
import math
import re
from pathlib import Path

import pytest

import paper_2609_33586_amd as pkg

HEADER = Path(__file__).resolve().parent.parent / "include" / "h15attn.h"


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", HEADER.read_text(), flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(attn_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    if not pkg.LIB_PATH.exists():
        from paper_2609_33586_amd import build
        build.build()
    return pkg.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) == set(pkg.EXPORTS)
    for n in names:
        assert hasattr(L, n)


def test_tile_and_strerror(L):
    assert pkg.attn_tile_bc() == 128
    assert pkg.attn_strerror(0) == "ok"
    for c in (-1, -2, -3, 7):
        assert isinstance(pkg.attn_strerror(c), str) and pkg.attn_strerror(c)


FAKE = 0x100000  # a 16-byte aligned address that is never dereferenced on error


def call(L, q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=None, B=1, Hq=2, Hkv=1, S=64, d=128, causal=0,
         scale=0.1, dtype=0, mode=1, opts=None):
    if opts is None:
        return L.attn_fwd_ex(q, k, v, o, lse, B, Hq, Hkv, S, d, causal, scale, dtype, mode, None)
    return L.attn_fwd_ex(q, k, v, o, lse, B, Hq, Hkv, S, d, causal, scale, dtype, mode, ctypes.byref(opts))


def test_invalid_arguments(L):
    E_INV, E_UNS = pkg.ATTN_EINVAL, pkg.ATTN_EUNSUPPORTED
    assert call(L, q=None) == E_INV
    assert call(L, o=None) == E_INV
    for kw in ({"B": 0}, {"Hq": 0}, {"Hkv": 0}, {"S": 0}, {"S": -5}, {"d": 0}):
        assert call(L, **kw) == E_INV
    assert call(L, Hq=3, Hkv=2) == E_INV
    for sc in (0.0, -1.0, math.inf, math.nan):
        assert call(L, scale=sc) == E_INV
    assert call(L, d=96) == E_UNS and call(L, d=256) == E_UNS
    assert call(L, dtype=2) == E_UNS and call(L, mode=5) == E_UNS
    assert call(L, q=FAKE + 8) == E_UNS
    assert call(L, lse=FAKE + 2) == E_UNS
    # size limits: B*Hq*S rows, and one head's K/V bytes within 31-bit offsets
    assert call(L, B=4, Hq=2, Hkv=1, S=1 << 27) == E_UNS
    assert call(L, B=1, Hq=1, Hkv=1, S=1 << 23, d=128, dtype=0) == E_UNS
    # FP8 needs positive finite descales
    assert call(L, dtype=1) == E_INV
    for bad in ((0.0, 1.0, 1.0), (1.0, -1.0, 1.0), (1.0, 1.0, math.inf)):
        assert call(L, dtype=1, opts=pkg.attn_opts(*bad, None)) == E_INV


def test_rescale_threshold_validation(L):
    E_INV, E_UNS = pkg.ATTN_EINVAL, pkg.ATTN_EUNSUPPORTED
    for tau in (-1.0, -1e-30, 64.5, math.inf, math.nan):
        assert call(L, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, tau, 0)) == E_INV
        assert call(L, dtype=1, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, tau, 1)) == E_INV
    # FP8 P must stay within e4m3's range: only tau = 0
    for tau in (0.5, 8.0):
        assert call(L, dtype=1, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, tau, 0)) == E_UNS


def test_rowmax_pot_is_bf16_only(L):
    E_UNS = pkg.ATTN_EUNSUPPORTED
    pot = pkg.ATTN_EXP_ROWMAX_POT
    assert call(L, dtype=1, mode=pot, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, 0.0, 0)) == E_UNS
    assert call(L, dtype=0, mode=pot, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, 8.0, 0)) == E_UNS
    assert call(L, mode=5) == E_UNS


def test_probe_invalid_rows(L):
    opts = pkg.attn_opts(1.0, 1.0, 1.0, None)
    args = [FAKE, FAKE, FAKE, FAKE, None, 1, 2, 1, 64, 128, 0, 0.1, 0, 1, ctypes.byref(opts)]
    for b, h, r0, n in ((1, 0, 0, 1), (0, 2, 0, 1), (0, 0, -1, 1), (0, 0, 0, 0), (0, 0, 60, 5)):
        assert L.attn_fwd_probe(*args, b, h, r0, n, FAKE, FAKE, FAKE) == pkg.ATTN_EINVAL
    assert L.attn_fwd_probe(*args, 0, 0, 0, 4, None, FAKE, FAKE) == pkg.ATTN_EINVAL


def test_attn_fwd_accepts_fp8_without_descales(L):
    # attn_fwd takes FP8 operands at unit descales: an FP8 call passes the
    # descale check and is stopped only by the size limit checked after it
    # (B*Hq*S beyond 2^30), before anything is launched; attn_fwd_ex without
    # options refuses FP8 for want of descales
    big = [FAKE, FAKE, FAKE, FAKE, None, 8, 2, 1, 1 << 27, 128, 0, 0.1, 1, 1]
    assert L.attn_fwd(*big) == pkg.ATTN_EUNSUPPORTED
    assert L.attn_fwd_ex(*big, None) == pkg.ATTN_EINVAL
    assert L.attn_fwd(None, *big[1:]) == pkg.ATTN_EINVAL


def dcall(L, q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=None, B=1, Hq=4, Hkv=2, Sq=1, Sk=1000, cap=1024, d=128,
          causal=1, scale=0.1, dtype=0, mode=1, split=0, ws=None, wsb=0, opts=None):
    return L.attn_decode(q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, cap, d, causal, scale, dtype, mode, split, ws, wsb,
                         ctypes.byref(opts) if opts is not None else None)


def test_decode_invalid_arguments(L):
    E_INV, E_UNS = pkg.ATTN_EINVAL, pkg.ATTN_EUNSUPPORTED
    assert dcall(L, q=None) == E_INV and dcall(L, o=None) == E_INV
    for kw in ({"B": 0}, {"Sq": 0}, {"Sk": 0}, {"cap": 0}, {"Hkv": 3}):
        assert dcall(L, **kw) == E_INV
    assert dcall(L, Sq=1001) == E_INV          # more query rows than keys
    assert dcall(L, Sk=1025) == E_INV          # beyond the cache
    assert dcall(L, split=100) == E_INV and dcall(L, split=-128) == E_INV
    assert dcall(L, d=96) == E_UNS and dcall(L, mode=pkg.ATTN_EXP_ROWMAX_POT) == E_UNS
    assert dcall(L, dtype=1) == E_INV          # FP8 needs descales
    assert dcall(L, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, 8.0, 0)) == E_UNS
    assert dcall(L, opts=pkg.attn_opts(1.0, 1.0, 1.0, None, -1.0, 0)) == E_INV
    assert dcall(L, q=FAKE + 8) == E_UNS
    assert dcall(L, cap=1 << 24, Sk=1 << 23) == E_UNS  # one head's cache beyond 31-bit offsets
    # several parts need a workspace of the stated size, 16-byte aligned
    need = pkg.attn_decode_workspace_bytes(1, 4, 1, 1000, 128, 256)
    assert need == 4 * 1 * 4 * (128 + 2) * 4  # rows x parts x (d + 2) floats
    assert dcall(L, split=256) == E_INV
    assert dcall(L, split=256, ws=FAKE, wsb=need - 1) == E_INV
    assert dcall(L, split=256, ws=FAKE + 4, wsb=need) == E_INV
    args = [FAKE, FAKE, FAKE, FAKE, None, 1, 4, 2, 2, 1000, 1024, 128, 1, 0.1, 0, 1, 0, None, 0, None]
    for b, h, i in ((1, 0, 0), (0, 4, 0), (0, 0, 2), (0, 0, -1)):
        assert L.attn_decode_probe(*args, b, h, i, FAKE, FAKE, FAKE) == E_INV
    assert L.attn_decode_probe(*args, 0, 0, 0, None, FAKE, FAKE) == E_INV


def test_decode_split_and_workspace_sizes(L):
    assert pkg.attn_decode_workspace_bytes(1, 4, 1, 1000, 128, 0) == 0       # one part
    assert pkg.attn_decode_workspace_bytes(1, 4, 1, 1000, 128, 1024) == 0    # one part
    assert pkg.attn_decode_workspace_bytes(2, 8, 3, 1000, 64, 128) == 2 * 8 * 3 * 8 * 66 * 4
    # the proposed cut: whole tiles, about 512 workgroups, at least eight tiles each
    assert pkg.attn_decode_split_keys(1, 32, 8, 1, 32768, 128, 0) == 1024    # 8 groups x 32 parts of 8 tiles
    assert pkg.attn_decode_split_keys(16, 32, 8, 1, 8192, 128, 1) == 2048    # 128 groups x 4 parts
    assert pkg.attn_decode_split_keys(64, 32, 8, 1, 4096, 128, 0) == 0       # 512 groups: no cut
    assert pkg.attn_decode_split_keys(1, 8, 8, 1, 600, 128, 0) == 0          # under eight tiles
    assert pkg.attn_decode_split_keys(0, 8, 8, 1, 600, 128, 0) == 0
    for args in ((1, 8, 1, 1, 100000, 128, 0), (3, 64, 8, 4, 5000, 64, 1)):
        s = pkg.attn_decode_split_keys(*args)
        assert s % 128 == 0 and s >= 0


def test_decode_noalloc_checks(L):
    # argument checks as attn_decode, then the built-in buffer's 16 MiB limit,
    # all before the GPU is touched
    E_INV = pkg.ATTN_EINVAL
    args = [FAKE, FAKE, FAKE, FAKE, None, 4, 64, 8, 1, 16384, 16384, 128, 1, 0.1, 0, 1]
    assert pkg.attn_decode_workspace_bytes(4, 64, 1, 16384, 128, 128) == 4 * 64 * 128 * 130 * 4 > 16 << 20
    assert L.attn_decode_noalloc(*args, 128, None) == pkg.ATTN_ENOSPACE
    assert L.attn_decode_noalloc(None, *args[1:], 128, None) == E_INV
    assert L.attn_decode_noalloc(*args, 100, None) == E_INV
    assert L.attn_decode_noalloc(*args[:9], 16385, *args[10:], 0, None) == E_INV  # Sk beyond the cache
    assert L.attn_decode_noalloc(*args[:14], 1, 1, 128, None) == E_INV  # FP8 without descales
    assert pkg.attn_strerror(pkg.ATTN_ENOSPACE) != pkg.attn_strerror(7)


def test_binding_checks_given_outputs():
    # the library writes through the data pointers it is given, so the
    # binding refuses output tensors it could not write as [B,Hq,S,d] bf16 /
    # [B,Hq,S] fp32 row-major (checked on host tensors: no GPU needed)
    import torch
    q = torch.zeros((2, 4, 40, 64), dtype=torch.bfloat16)
    good_o = torch.empty((2, 4, 40, 64), dtype=torch.bfloat16)
    good_l = torch.empty((2, 4, 40), dtype=torch.float32)
    o, l = pkg._outputs(q, good_o, good_l, True)
    assert o is good_o and l is good_l
    assert pkg._outputs(q, good_o, None, False)[1] is None
    bad_o = [torch.empty((2, 4, 40, 128), dtype=torch.bfloat16),             # shape
             torch.empty((2, 4, 40, 64), dtype=torch.float32),               # type
             torch.empty((2, 4, 64, 40), dtype=torch.bfloat16).transpose(2, 3)]  # not contiguous
    for t in bad_o:
        with pytest.raises(ValueError):
            pkg._outputs(q, t, good_l, True)
    bad_l = [torch.empty((2, 4, 41), dtype=torch.float32), torch.empty((2, 4, 40), dtype=torch.bfloat16),
             torch.empty((2, 40, 4), dtype=torch.float32).transpose(1, 2)]
    for t in bad_l:
        with pytest.raises(ValueError):
            pkg._outputs(q, good_o, t, True)
    ws = torch.empty((64, 2), dtype=torch.uint8).t()
    with pytest.raises(ValueError):
        pkg._workspace(q, 2, 4, 40, 1000, 64, 128, ws)


def test_library_links_both_kernel_units(L):
    # the kernel file is compiled twice (the FP8 lattice-weight forward at
    # d = 128 on its own): the library must hold that unit's launcher and
    # exactly one launch stub per forward kernel instantiation
    import subprocess
    out = subprocess.run(["nm", "-C", str(pkg.LIB_PATH)], capture_output=True, text=True, check=True).stdout
    assert re.search(r"\bT h15::launch_fwd_fp8_lattice128\(", out)
    stubs = re.findall(r"__device_stub__attn_fwd_kernel<(\d), (\d+), (true|false), (\d), (true|false), (true|false)>",
                       out)
    assert len(stubs) == len(set(stubs))
    lattice128 = {s for s in stubs if s[0] == "1" and s[1] == "128" and s[3] != "0"}
    assert len(lattice128) == 2 * 6 * 2  # causal x the six lattice modes x probe
    # BF16: d x causal x probe x (5 default + 4 compact); FP8: d x causal x probe x 7 modes
    assert len(stubs) == 2 * 2 * 2 * 9 + 2 * 2 * 2 * 7
