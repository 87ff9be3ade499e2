"""Rowmax-H15 fused attention forward for MI355X (gfx950).

A thin ctypes binding over ``libh15attn.so`` (built from ``csrc/h15attn.hip``
by ``build.py``).  Every step of the attention runs in the HIP kernels; this
module only marshals torch tensors (device memory and streams) into the C ABI
declared in ``include/h15attn.h``.  The functions carry the C names.

There is no fallback: if the library is missing or a call fails, an exception
is raised.
"""
from __future__ import annotations

import ctypes
import os
from pathlib import Path

_PKG = Path(__file__).resolve().parent
LIB_PATH = _PKG / "libh15attn.so"

ATTN_BF16, ATTN_FP8_E4M3 = 0, 1
ATTN_EXP_EXACT, ATTN_EXP_H15, ATTN_EXP_SQ4, ATTN_EXP_SQ8, ATTN_EXP_ROWMAX_POT = 0, 1, 2, 3, 4
ATTN_OK, ATTN_EINVAL, ATTN_EUNSUPPORTED, ATTN_ELAUNCH, ATTN_ENOSPACE = 0, -1, -2, -3, -4

# every symbol the header declares
EXPORTS = ("attn_fwd", "attn_fwd_ex", "attn_fwd_probe", "attn_strerror", "attn_tile_bc", "attn_decode",
           "attn_decode_workspace_bytes", "attn_decode_split_keys", "attn_decode_probe", "attn_decode_noalloc")


class attn_opts(ctypes.Structure):
    _fields_ = [("q_descale", ctypes.c_float), ("k_descale", ctypes.c_float),
                ("v_descale", ctypes.c_float), ("stream", ctypes.c_void_p),
                ("rescale_threshold", ctypes.c_float), ("rescale_per_wave", ctypes.c_int)]


class AttnError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where}: {attn_strerror(code)} ({code})")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load libh15attn.so (raises if it has not been built).  H15ATTN_LIB, when
    set, names another build of the library to load instead (the host-only
    sanitizer build of the argument checks)."""
    global _lib
    if _lib is not None:
        return _lib
    path = Path(os.environ.get("H15ATTN_LIB", "") or LIB_PATH)
    if not path.exists():
        raise RuntimeError(f"{path} is missing: build it with paper_2609_33586_amd.build.build()")
    L = ctypes.CDLL(str(path))
    P, I, F = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
    common = [P, P, P, P, P, I, I, I, I, I, I, F, I, I]
    L.attn_fwd.argtypes = common
    L.attn_fwd.restype = I
    L.attn_fwd_ex.argtypes = common + [ctypes.POINTER(attn_opts)]
    L.attn_fwd_ex.restype = I
    L.attn_fwd_probe.argtypes = common + [ctypes.POINTER(attn_opts), I, I, I, I, P, P, P]
    L.attn_fwd_probe.restype = I
    L.attn_strerror.argtypes = [I]
    L.attn_strerror.restype = ctypes.c_char_p
    L.attn_tile_bc.argtypes = []
    L.attn_tile_bc.restype = I
    dec = [P, P, P, P, P, I, I, I, I, I, I, I, I, F, I, I, I, P, ctypes.c_size_t, ctypes.POINTER(attn_opts)]
    L.attn_decode.argtypes = dec
    L.attn_decode.restype = I
    L.attn_decode_noalloc.argtypes = dec[:17] + [ctypes.POINTER(attn_opts)]
    L.attn_decode_noalloc.restype = I
    L.attn_decode_probe.argtypes = dec + [I, I, I, P, P, P]
    L.attn_decode_probe.restype = I
    L.attn_decode_workspace_bytes.argtypes = [I, I, I, I, I, I]
    L.attn_decode_workspace_bytes.restype = ctypes.c_size_t
    L.attn_decode_split_keys.argtypes = [I, I, I, I, I, I, I]
    L.attn_decode_split_keys.restype = I
    _lib = L
    return L


def attn_strerror(code: int) -> str:
    return lib().attn_strerror(int(code)).decode()


def attn_tile_bc() -> int:
    return int(lib().attn_tile_bc())


def _dtype_of(t) -> int:
    import torch
    if t.dtype in (torch.bfloat16, torch.uint16, torch.int16):
        return ATTN_BF16
    if t.dtype in (torch.float8_e4m3fn, torch.uint8):
        return ATTN_FP8_E4M3
    raise TypeError(f"unsupported operand dtype {t.dtype}")


def _check(q, k, v):
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
            raise ValueError(f"{name} must be a contiguous 4-D device tensor [B,H,S,d]")
    B, Hq, S, d = q.shape
    Hkv = k.shape[1]
    if tuple(k.shape) != (B, Hkv, S, d) or tuple(v.shape) != (B, Hkv, S, d):
        raise ValueError("k and v must be [B,Hkv,S,d] with q's B, S, d")
    dt = _dtype_of(q)
    if _dtype_of(k) != dt or _dtype_of(v) != dt:
        raise TypeError("q, k, v must share one operand type")
    return B, Hq, Hkv, S, d, dt


def _outputs(q, out, lse, want_lse):
    """O [B,Hq,S,d] bf16 and LSE [B,Hq,S] fp32 (None unless wanted or given):
    the caller's tensors after checks, else new ones.  The library writes
    through the data pointers, so a given tensor must be contiguous, of the
    right shape and type, and on q's device."""
    import torch
    B, Hq, S, d = q.shape
    if out is None:
        out = torch.empty((B, Hq, S, d), dtype=torch.bfloat16, device=q.device)
    elif (tuple(out.shape) != (B, Hq, S, d) or out.dtype != torch.bfloat16 or not out.is_contiguous()
          or out.device != q.device):
        raise ValueError(f"out must be a contiguous bfloat16 tensor {(B, Hq, S, d)} on {q.device}")
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, S), dtype=torch.float32, device=q.device)
    elif lse is not None and (tuple(lse.shape) != (B, Hq, S) or lse.dtype != torch.float32
                              or not lse.is_contiguous() or lse.device != q.device):
        raise ValueError(f"lse must be a contiguous float32 tensor {(B, Hq, S)} on {q.device}")
    return out, lse


def _opts(descale, stream, tau=0.0, tau_per_wave=False):
    import torch
    qd, kd, vd = descale if descale is not None else (1.0, 1.0, 1.0)
    st = stream if stream is not None else torch.cuda.current_stream()
    return attn_opts(float(qd), float(kd), float(vd), ctypes.c_void_p(st.cuda_stream), float(tau),
                     int(bool(tau_per_wave)))


def attn_fwd_ex(q, k, v, *, causal: bool, scale: float, exp_mode: int, descale=None, stream=None,
                out=None, lse=None, want_lse: bool = True, tau: float = 0.0, tau_per_wave: bool = False):
    """O (and LSE) of attention; see include/h15attn.h for the definition.
    tau / tau_per_wave: the conditional-rescale threshold and its granularity."""
    B, Hq, Hkv, S, d, dt = _check(q, k, v)
    out, lse = _outputs(q, out, lse, want_lse)
    opts = _opts(descale, stream, tau, tau_per_wave)
    rc = lib().attn_fwd_ex(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                           lse.data_ptr() if lse is not None else None, B, Hq, Hkv, S, d,
                           int(bool(causal)), float(scale), dt, int(exp_mode), ctypes.byref(opts))
    if rc != ATTN_OK:
        raise AttnError(rc, "attn_fwd_ex")
    return out, lse


def attn_fwd(q, k, v, *, causal: bool, scale: float, exp_mode: int, out=None, lse=None,
             want_lse: bool = True):
    """attn_fwd on the default stream with unit descales."""
    B, Hq, Hkv, S, d, dt = _check(q, k, v)
    out, lse = _outputs(q, out, lse, want_lse)
    rc = lib().attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                        lse.data_ptr() if lse is not None else None, B, Hq, Hkv, S, d,
                        int(bool(causal)), float(scale), dt, int(exp_mode))
    if rc != ATTN_OK:
        raise AttnError(rc, "attn_fwd")
    return out, lse


def attn_fwd_probe(q, k, v, *, causal: bool, scale: float, exp_mode: int, b: int, h: int,
                   row0: int, nrows: int, descale=None, stream=None, tau: float = 0.0,
                   tau_per_wave: bool = False):
    """Returns (O, LSE, s, w, p_bits) with s/w/p_bits of shape [nrows, S]."""
    import torch
    B, Hq, Hkv, S, d, dt = _check(q, k, v)
    out, lse = _outputs(q, None, None, True)
    s = torch.empty((nrows, S), dtype=torch.float32, device=q.device)
    w = torch.empty((nrows, S), dtype=torch.float32, device=q.device)
    pb = torch.empty((nrows, S), dtype=torch.int32, device=q.device)
    opts = _opts(descale, stream, tau, tau_per_wave)
    rc = lib().attn_fwd_probe(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                              B, Hq, Hkv, S, d, int(bool(causal)), float(scale), dt, int(exp_mode),
                              ctypes.byref(opts), int(b), int(h), int(row0), int(nrows),
                              s.data_ptr(), w.data_ptr(), pb.data_ptr())
    if rc != ATTN_OK:
        raise AttnError(rc, "attn_fwd_probe")
    return out, lse, s, w, pb


# ---- decode over a key/value cache ------------------------------------------

def attn_decode_split_keys(B: int, Hq: int, Hkv: int, Sq: int, Sk: int, d: int, dtype: int) -> int:
    """The library's proposed key cut for attn_decode (0: one part)."""
    return int(lib().attn_decode_split_keys(int(B), int(Hq), int(Hkv), int(Sq), int(Sk), int(d), int(dtype)))


def attn_decode_workspace_bytes(B: int, Hq: int, Sq: int, Sk: int, d: int, split_keys: int) -> int:
    return int(lib().attn_decode_workspace_bytes(int(B), int(Hq), int(Sq), int(Sk), int(d), int(split_keys)))


def _check_decode(q, k, v, Sk):
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
            raise ValueError(f"{name} must be a contiguous 4-D device tensor")
    B, Hq, Sq, d = q.shape
    Hkv, cap = k.shape[1], k.shape[2]
    if tuple(k.shape) != (B, Hkv, cap, d) or tuple(v.shape) != tuple(k.shape):
        raise ValueError("k and v must be [B,Hkv,Sk_cap,d] with q's B and d")
    dt = _dtype_of(q)
    if _dtype_of(k) != dt or _dtype_of(v) != dt:
        raise TypeError("q, k, v must share one operand type")
    return B, Hq, Hkv, Sq, (cap if Sk is None else int(Sk)), cap, d, dt


def _workspace(q, B, Hq, Sq, Sk, d, split_keys, workspace):
    import torch
    need = attn_decode_workspace_bytes(B, Hq, Sq, Sk, d, split_keys)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device) if need else None
    elif not workspace.is_contiguous() or workspace.device != q.device:
        raise ValueError(f"workspace must be a contiguous tensor on {q.device}")
    ptr = workspace.data_ptr() if workspace is not None else None
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    return workspace, ptr, nbytes


def attn_decode(q, k, v, *, causal: bool, scale: float, exp_mode: int, split_keys: int, Sk: int | None = None,
                descale=None, stream=None, out=None, lse=None, want_lse: bool = True, workspace=None):
    """Decode over a key/value cache (see include/h15attn.h, attn_decode).

    q: [B,Hq,Sq,d]; k, v: [B,Hkv,Sk_cap,d] whose first Sk rows (default all)
    are the cache.  Returns (O [B,Hq,Sq,d] bf16, LSE [B,Hq,Sq] fp32 or None).
    workspace: a device buffer of attn_decode_workspace_bytes() bytes
    (allocated here when None and the cut has several parts)."""
    B, Hq, Hkv, Sq, Sk, cap, d, dt = _check_decode(q, k, v, Sk)
    out, lse = _outputs(q, out, lse, want_lse)
    ws, wptr, wbytes = _workspace(q, B, Hq, Sq, Sk, d, split_keys, workspace)
    opts = _opts(descale, stream)
    rc = lib().attn_decode(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                           lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Sq, Sk, cap, d,
                           int(bool(causal)), float(scale), dt, int(exp_mode), int(split_keys), wptr, wbytes,
                           ctypes.byref(opts))
    if rc != ATTN_OK:
        raise AttnError(rc, "attn_decode")
    return out, lse


def attn_decode_noalloc(q, k, v, *, causal: bool, scale: float, exp_mode: int, split_keys: int,
                        Sk: int | None = None, descale=None, stream=None, out=None, lse=None, want_lse: bool = True):
    """attn_decode with the library's built-in workspace (see include/h15attn.h,
    attn_decode_noalloc).  Pass out (and lse) to keep the call free of
    allocations; calls that overlap on one GPU race on the built-in buffer."""
    B, Hq, Hkv, Sq, Sk, cap, d, dt = _check_decode(q, k, v, Sk)
    out, lse = _outputs(q, out, lse, want_lse)
    opts = _opts(descale, stream)
    rc = lib().attn_decode_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                                   lse.data_ptr() if lse is not None else None, B, Hq, Hkv, Sq, Sk, cap, d,
                                   int(bool(causal)), float(scale), dt, int(exp_mode), int(split_keys),
                                   ctypes.byref(opts))
    if rc != ATTN_OK:
        raise AttnError(rc, "attn_decode_noalloc")
    return out, lse


def attn_decode_probe(q, k, v, *, causal: bool, scale: float, exp_mode: int, split_keys: int, b: int, h: int,
                      i: int, Sk: int | None = None, descale=None, stream=None):
    """Returns (O, LSE, s, w, p_bits) with s/w/p_bits of shape [Sk] for query row (b, h, i)."""
    import torch
    B, Hq, Hkv, Sq, Sk, cap, d, dt = _check_decode(q, k, v, Sk)
    out, lse = _outputs(q, None, None, True)
    ws, wptr, wbytes = _workspace(q, B, Hq, Sq, Sk, d, split_keys, None)
    s = torch.empty(Sk, dtype=torch.float32, device=q.device)
    w = torch.empty(Sk, dtype=torch.float32, device=q.device)
    pb = torch.empty(Sk, dtype=torch.int32, device=q.device)
    opts = _opts(descale, stream)
    rc = lib().attn_decode_probe(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(), B, Hq,
                                 Hkv, Sq, Sk, cap, d, int(bool(causal)), float(scale), dt, int(exp_mode),
                                 int(split_keys), wptr, wbytes, ctypes.byref(opts), int(b), int(h), int(i),
                                 s.data_ptr(), w.data_ptr(), pb.data_ptr())
    if rc != ATTN_OK:
        raise AttnError(rc, "attn_decode_probe")
    return out, lse, s, w, pb
