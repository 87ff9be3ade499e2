"""CPU oracle for softmax attention and Rowmax-H15 attention (test infrastructure).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
and the CPU-baseline leg of the benchmark may import this package.  It shares
no code with the GPU library; the arithmetic lives in ``attn_oracle.c`` (plain
C, fp64 accumulation), this module only marshals numpy arrays through ctypes.

Paper: "Approximating Softmax in Pretrained LLMs: Model Sensitivity and Kernel
Acceleration".  Modes follow App. A.1 Eq. (exact-attention) (EXACT),
Sec. 5.2 Eq. (m-h15) with App. B.1 "Implementation" and the per-tile running
max of App. B.2 (H15_TILE), the whole-row control of Table B2 (H15_WHOLEROW),
App. A.6 Eq. (rowmax-pot) (ROWMAX_POT) and the finer input-rounding family
S(Q_{2^-k}(x)) of App. B.2 "Exponential-map ablation" with the per-tile running
max (SQ4_TILE for k = 2, SQ8_TILE for k = 3).
"""
from __future__ import annotations

import ctypes
import os
from pathlib import Path

import numpy as np

from .build import build as _build, LIB_PATH

BF16, FP8_E4M3 = 0, 1
EXACT, H15_TILE, H15_WHOLEROW, ROWMAX_POT, EXACT_TILE, SQ4_TILE, SQ8_TILE = 0, 1, 2, 3, 4, 5, 6
# input-rounding exponent k of each tiled mode (Rowmax-H15 is k = 1)
MODE_K = {H15_TILE: 1, H15_WHOLEROW: 1, SQ4_TILE: 2, SQ8_TILE: 3}

_lib = None


def lib() -> ctypes.CDLL:
    """Load the oracle library, building it first when it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    path = Path(os.environ.get("H15_ORACLE_LIB", "") or LIB_PATH)  # a sanitizer build, when set
    if not path.exists():
        if path != LIB_PATH:
            raise RuntimeError(f"H15_ORACLE_LIB={path} does not exist")
        _build()
    L = ctypes.CDLL(str(path))
    c_f, c_d, c_i, c_i64, c_p = ctypes.c_float, ctypes.c_double, ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
    L.oracle_threads.restype = c_i
    L.oracle_bf16_value.argtypes = [ctypes.c_uint16]
    L.oracle_bf16_value.restype = c_d
    L.oracle_e4m3_value.argtypes = [ctypes.c_uint8]
    L.oracle_e4m3_value.restype = c_d
    L.oracle_e4m3_rne_satfinite.argtypes = [c_d]
    L.oracle_e4m3_rne_satfinite.restype = ctypes.c_uint8
    L.oracle_h15_weight.argtypes = [c_f]
    L.oracle_h15_weight.restype = c_f
    L.oracle_h15_ideal.argtypes = [c_d]
    L.oracle_h15_ideal.restype = c_d
    L.oracle_h15_exhaustive.argtypes = [c_f, c_f, ctypes.POINTER(c_i64)]
    L.oracle_h15_exhaustive.restype = c_i64
    L.oracle_sq_weight.argtypes = [c_f, c_i]
    L.oracle_sq_weight.restype = c_f
    L.oracle_sq_ideal.argtypes = [c_d, c_i]
    L.oracle_sq_ideal.restype = c_d
    L.oracle_sq_exhaustive.argtypes = [c_f, c_f, c_i, ctypes.POINTER(c_i64)]
    L.oracle_sq_exhaustive.restype = c_i64
    L.oracle_sq_count_mismatch.argtypes = [c_p, c_i64, c_i]
    L.oracle_sq_count_mismatch.restype = c_i64
    L.oracle_sq_row_from_logits.argtypes = [c_p, c_i, c_i, c_i, c_f, c_i, c_i, c_d, c_i, c_i, c_p, c_p, c_p]
    L.oracle_sq_row_from_logits.restype = c_i
    L.oracle_pot_row_from_logits.argtypes = [c_p, c_i, c_i, c_i, c_f, c_p, c_p, c_p]
    L.oracle_pot_row_from_logits.restype = c_i
    L.oracle_c1.argtypes = [c_d, c_d, c_d]
    L.oracle_c1.restype = c_f
    L.oracle_h15_row_from_logits.argtypes = [c_p, c_i, c_i, c_i, c_f, c_i, c_i, c_d, c_i, c_p, c_p, c_p]
    L.oracle_h15_row_from_logits.restype = c_i
    L.oracle_attn.argtypes = [c_p, c_p, c_p, c_i, c_d, c_d, c_d, c_i, c_i, c_i, c_i, c_i, c_i, c_d,
                              c_i, c_i, c_d, c_i, c_p, c_i64, c_p, c_p]
    L.oracle_group_moves_from_logits.argtypes = [c_p, c_i, c_i, c_i, c_i, c_f, c_i, c_d, c_p]
    L.oracle_group_moves_from_logits.restype = c_i
    L.oracle_sq_row_from_logits_moves.argtypes = [c_p, c_i, c_i, c_i, c_f, c_i, c_i, c_p, c_i, c_p, c_p, c_p]
    L.oracle_sq_row_from_logits_moves.restype = c_i
    L.oracle_attn.restype = c_i
    L.oracle_logits_row.argtypes = [c_p, c_p, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_p]
    L.oracle_logits_row.restype = c_i
    L.oracle_sq_row_exponents_from_logits.argtypes = [c_p, c_i, c_i, c_i, c_f, c_i, c_i, c_i, c_i, c_p, c_p, c_p]
    L.oracle_sq_row_exponents_from_logits.restype = c_i
    L.oracle_decode.argtypes = [c_p, c_p, c_p, c_i, c_d, c_d, c_d, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_d,
                                c_i, c_i, c_i, c_p, c_i64, c_p, c_p]
    L.oracle_decode.restype = c_i
    L.oracle_decode_row_from_logits.argtypes = [c_p, c_i, c_i, c_f, c_i, c_i, c_i, c_i, c_i, c_p, c_p, c_p]
    L.oracle_decode_row_from_logits.restype = c_i
    L.oracle_decode_logits_row.argtypes = [c_p, c_p, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_i, c_p]
    L.oracle_decode_logits_row.restype = c_i
    _lib = L
    return L


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def threads() -> int:
    return lib().oracle_threads()


def bf16_value(bits: int) -> float:
    return lib().oracle_bf16_value(int(bits))


def e4m3_value(code: int) -> float:
    return lib().oracle_e4m3_value(int(code))


def e4m3_encode(x: float) -> int:
    return int(lib().oracle_e4m3_rne_satfinite(float(x)))


def h15_weight(y: float) -> float:
    """App. B.1 FP32 add/shift realisation on the doubled exponent y = 2x."""
    return lib().oracle_h15_weight(float(y))


def h15_ideal(y: float) -> float:
    """Eq. (m-h15) closed form on the doubled exponent y = 2x (no clamp)."""
    return lib().oracle_h15_ideal(float(y))


def h15_exhaustive(lo: float, hi: float) -> tuple[int, int]:
    """Compare the two forms over every fp32 value in [lo, hi]; (mismatches, count)."""
    n = ctypes.c_int64(0)
    bad = lib().oracle_h15_exhaustive(float(lo), float(hi), ctypes.byref(n))
    return int(bad), int(n.value)


def sq_weight(y: float, k: int) -> float:
    """S(Q_{2^-k}) realisation (App. B.2 ablation): add 0x4B400000, shift by 23 - k; y = 2^k x."""
    return lib().oracle_sq_weight(float(y), int(k))


def sq_ideal(y: float, k: int) -> float:
    """S(Q_{2^-k}(x)) from the definitions of S and Q, on y = 2^k x (no clamp)."""
    return lib().oracle_sq_ideal(float(y), int(k))


def sq_exhaustive(lo: float, hi: float, k: int) -> tuple[int, int]:
    """Compare the two forms over every fp32 value in [lo, hi]; (mismatches, count)."""
    n = ctypes.c_int64(0)
    bad = lib().oracle_sq_exhaustive(float(lo), float(hi), int(k), ctypes.byref(n))
    return int(bad), int(n.value)


def sq_count_mismatch(x: np.ndarray, k: int) -> int:
    """Realisation vs S(Q_{2^-k}) on base-two exponents x (clamped at -126); mismatches."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return int(lib().oracle_sq_count_mismatch(_ptr(x), int(x.shape[0]), int(k)))


def c1(scale: float, qd: float = 1.0, kd: float = 1.0) -> float:
    """Base-two exponent scale of a raw logit, fp32(scale*qd*kd*log2 e)."""
    return lib().oracle_c1(float(scale), float(qd), float(kd))


def h15_row_from_logits(s: np.ndarray, i: int, causal: bool, c1_: float, dtype: int,
                        Bc: int, tau: float = 0.0, exact_exp: bool = False):
    """W (fp32) and P bits (bf16 or e4m3 code) of query row i from its fp32 logits.

    Returns (W, P, lse)."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    S = s.shape[0]
    w = np.zeros(S, np.float32)
    p = np.zeros(S, np.uint32)
    lse = ctypes.c_double(0.0)
    rc = lib().oracle_h15_row_from_logits(_ptr(s), S, int(i), int(bool(causal)), float(c1_), int(dtype),
                                          int(Bc), float(tau), int(bool(exact_exp)), _ptr(w), _ptr(p),
                                          ctypes.byref(lse))
    if rc != 0:
        raise ValueError("oracle_h15_row_from_logits: invalid arguments")
    return w, p, lse.value


def sq_row_from_logits(s: np.ndarray, i: int, causal: bool, c1_: float, dtype: int, Bc: int, k: int,
                       tau: float = 0.0):
    """As h15_row_from_logits for the weight S(Q_{2^-k}) (k = 1 is Rowmax-H15)."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    S = s.shape[0]
    w = np.zeros(S, np.float32)
    p = np.zeros(S, np.uint32)
    lse = ctypes.c_double(0.0)
    rc = lib().oracle_sq_row_from_logits(_ptr(s), S, int(i), int(bool(causal)), float(c1_), int(dtype),
                                         int(Bc), float(tau), 0, int(k), _ptr(w), _ptr(p), ctypes.byref(lse))
    if rc != 0:
        raise ValueError("oracle_sq_row_from_logits: invalid arguments")
    return w, p, lse.value


def group_moves_from_logits(s: np.ndarray, i0: int, causal: bool, c1_: float, Bc: int, tau: float) -> np.ndarray:
    """Per-tile anchor decisions shared by the rows i0 .. i0 + len(s) - 1, from
    their fp32 logits s [rows, S] (1: move every row's anchor to its max)."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    n, S = s.shape
    move = np.zeros(S // Bc + 1, np.uint8)
    rc = lib().oracle_group_moves_from_logits(_ptr(s), S, int(i0), int(i0 + n), int(bool(causal)), float(c1_),
                                              int(Bc), float(tau), _ptr(move))
    if rc != 0:
        raise ValueError("oracle_group_moves_from_logits: invalid arguments")
    return move


def sq_row_from_logits_moves(s: np.ndarray, i: int, causal: bool, c1_: float, dtype: int, Bc: int, k: int,
                             move: np.ndarray):
    """As sq_row_from_logits with the per-tile anchor decisions given."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    move = np.ascontiguousarray(move, dtype=np.uint8)
    S = s.shape[0]
    w = np.zeros(S, np.float32)
    p = np.zeros(S, np.uint32)
    lse = ctypes.c_double(0.0)
    rc = lib().oracle_sq_row_from_logits_moves(_ptr(s), S, int(i), int(bool(causal)), float(c1_), int(dtype),
                                               int(Bc), _ptr(move), int(k), _ptr(w), _ptr(p), ctypes.byref(lse))
    if rc != 0:
        raise ValueError("oracle_sq_row_from_logits_moves: invalid arguments")
    return w, p, lse.value


def pot_row_from_logits(s: np.ndarray, i: int, causal: bool, c1_: float):
    """Rowmax-PoT (Eq. (rowmax-pot), K_max = 20) W, P (bf16 bits) and LSE of row i from fp32 logits."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    S = s.shape[0]
    w = np.zeros(S, np.float32)
    p = np.zeros(S, np.uint32)
    lse = ctypes.c_double(0.0)
    rc = lib().oracle_pot_row_from_logits(_ptr(s), S, int(i), int(bool(causal)), float(c1_), _ptr(w), _ptr(p),
                                          ctypes.byref(lse))
    if rc != 0:
        raise ValueError("oracle_pot_row_from_logits: invalid arguments")
    return w, p, lse.value


def attn(q: np.ndarray, k: np.ndarray, v: np.ndarray, *, dtype: int, causal: bool, scale: float,
         mode: int, descale=(1.0, 1.0, 1.0), Bc: int = 128, tau: float = 0.0, tau_group: int = 1,
         rows: np.ndarray | None = None):
    """Attention forward on stored operands.

    q: [B,Hq,S,d], k/v: [B,Hkv,S,d]; uint16 bf16 bit patterns (dtype BF16) or
    uint8 e4m3 codes (dtype FP8_E4M3).  tau: conditional-rescale threshold in
    base-two units (0: the anchor is always the running max); tau_group: rows
    per shared anchor decision (1: per row; 32: per aligned group of 32 rows,
    as FlashAttention-4 decides per warp).  rows: optional flat row indices
    (b*Hq + h)*S + i.  Returns (O [nrows, d] float64, LSE [nrows] float64);
    without rows the shapes are [B,Hq,S,d] and [B,Hq,S]."""
    want = np.uint16 if dtype == BF16 else np.uint8
    q = np.ascontiguousarray(q, dtype=want)
    k = np.ascontiguousarray(k, dtype=want)
    v = np.ascontiguousarray(v, dtype=want)
    B, Hq, S, d = q.shape
    Hkv = k.shape[1]
    if k.shape != (B, Hkv, S, d) or v.shape != k.shape:
        raise ValueError("shape mismatch")
    if rows is None:
        nrows = B * Hq * S
        rows_arr = None
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
        nrows = rows_arr.shape[0]
    o = np.zeros((nrows, d), np.float64)
    lse = np.zeros(nrows, np.float64)
    qd, kd, vd = (float(x) for x in descale)
    rc = lib().oracle_attn(_ptr(q), _ptr(k), _ptr(v), int(dtype), qd, kd, vd, B, Hq, Hkv, S, d,
                           int(bool(causal)), float(scale), int(mode), int(Bc), float(tau), int(tau_group),
                           _ptr(rows_arr), int(nrows), _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle_attn: out of memory" if rc == -3 else "oracle_attn: invalid arguments")
    if rows is None:
        return o.reshape(B, Hq, S, d), lse.reshape(B, Hq, S)
    return o, lse


def logits_row(q: np.ndarray, k: np.ndarray, dtype: int, b: int, h: int, i: int) -> np.ndarray:
    """fp32 raw logits of one query row (exact fp64 dot, rounded once)."""
    want = np.uint16 if dtype == BF16 else np.uint8
    q = np.ascontiguousarray(q, dtype=want)
    k = np.ascontiguousarray(k, dtype=want)
    B, Hq, S, d = q.shape
    out = np.zeros(S, np.float32)
    rc = lib().oracle_logits_row(_ptr(q), _ptr(k), int(dtype), B, Hq, k.shape[1], S, d, b, h, i, _ptr(out))
    if rc != 0:
        raise ValueError("oracle_logits_row: invalid arguments")
    return out


def row_exponents_from_logits(s: np.ndarray, i: int, causal: bool, c1_: float, dtype: int, Bc: int, k: int = 1,
                              exact_exp: bool = False):
    """Per-key exponent arguments of row i from fp32 logits: (y, anchor, W).

    y[j] is the fp32 value key j's weight is taken from (2^k x for the lattice
    weights, x for the exact exponential, before the clamp), anchor[j] the
    running max of its tile; masked keys have -inf in both."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    S = s.shape[0]
    y = np.zeros(S, np.float32)
    a = np.zeros(S, np.float32)
    w = np.zeros(S, np.float32)
    rc = lib().oracle_sq_row_exponents_from_logits(_ptr(s), S, int(i), int(bool(causal)), float(c1_), int(dtype),
                                                   int(Bc), int(bool(exact_exp)), int(k), _ptr(y), _ptr(a), _ptr(w))
    if rc != 0:
        raise ValueError("oracle_sq_row_exponents_from_logits: invalid arguments")
    return y, a, w


def decode(q: np.ndarray, k: np.ndarray, v: np.ndarray, *, Sk: int, dtype: int, causal: bool, scale: float,
           mode: int, split_keys: int, descale=(1.0, 1.0, 1.0), Bc: int = 128, rows: np.ndarray | None = None):
    """Decode attention over a key/value cache (see oracle_decode in attn_oracle.c).

    q: [B,Hq,Sq,d]; k/v: [B,Hkv,Sk_cap,d] whose first Sk rows per head are the
    cache.  Query i sees keys j <= Sk - Sq + i when causal.  The keys are cut
    into parts of split_keys (a multiple of Bc; 0: one part), each running the
    per-tile recurrence on its own, merged exactly.  Returns (O [nrows, d],
    LSE [nrows]) or, without rows, [B,Hq,Sq,d] and [B,Hq,Sq]."""
    want = np.uint16 if dtype == BF16 else np.uint8
    q = np.ascontiguousarray(q, dtype=want)
    k = np.ascontiguousarray(k, dtype=want)
    v = np.ascontiguousarray(v, dtype=want)
    B, Hq, Sq, d = q.shape
    Hkv, Sk_cap = k.shape[1], k.shape[2]
    if k.shape != (B, Hkv, Sk_cap, d) or v.shape != k.shape:
        raise ValueError("shape mismatch")
    if rows is None:
        nrows, rows_arr = B * Hq * Sq, None
    else:
        rows_arr = np.ascontiguousarray(rows, dtype=np.int64)
        nrows = rows_arr.shape[0]
    o = np.zeros((nrows, d), np.float64)
    lse = np.zeros(nrows, np.float64)
    qd, kd, vd = (float(x) for x in descale)
    rc = lib().oracle_decode(_ptr(q), _ptr(k), _ptr(v), int(dtype), qd, kd, vd, B, Hq, Hkv, Sq, int(Sk), Sk_cap, d,
                             int(bool(causal)), float(scale), int(mode), int(Bc), int(split_keys), _ptr(rows_arr),
                             int(nrows), _ptr(o), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle_decode: out of memory" if rc == -3 else "oracle_decode: invalid arguments")
    if rows is None:
        return o.reshape(B, Hq, Sq, d), lse.reshape(B, Hq, Sq)
    return o, lse


def decode_row_from_logits(s: np.ndarray, jend: int, c1_: float, dtype: int, Bc: int, split_keys: int, k: int = 1,
                           exact_exp: bool = False):
    """W, P bits and LSE of one decode row from its fp32 logits (jend visible keys)."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    Sk = s.shape[0]
    w = np.zeros(Sk, np.float32)
    p = np.zeros(Sk, np.uint32)
    lse = ctypes.c_double(0.0)
    rc = lib().oracle_decode_row_from_logits(_ptr(s), Sk, int(jend), float(c1_), int(dtype), int(Bc),
                                             int(split_keys), int(bool(exact_exp)), int(k), _ptr(w), _ptr(p),
                                             ctypes.byref(lse))
    if rc != 0:
        raise ValueError("oracle_decode_row_from_logits: invalid arguments")
    return w, p, lse.value


def decode_logits_row(q: np.ndarray, k: np.ndarray, dtype: int, Sk: int, b: int, h: int, i: int) -> np.ndarray:
    """fp32 raw logits of one decode row against the first Sk cache rows."""
    want = np.uint16 if dtype == BF16 else np.uint8
    q = np.ascontiguousarray(q, dtype=want)
    k = np.ascontiguousarray(k, dtype=want)
    B, Hq, Sq, d = q.shape
    out = np.zeros(int(Sk), np.float32)
    rc = lib().oracle_decode_logits_row(_ptr(q), _ptr(k), int(dtype), B, Hq, k.shape[1], Sq, int(Sk), k.shape[2], d,
                                        int(b), int(h), int(i), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_decode_logits_row: invalid arguments")
    return out
