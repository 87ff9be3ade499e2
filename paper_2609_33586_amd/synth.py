"""Seeded synthetic attention inputs (shared by the tests, the benchmark and the
CPU oracle's callers).

Holds no arithmetic of the attention method: it only draws Gaussian Q/K/V,
optionally makes 2% of the key positions "sharp" (x4), and stores them in
the operand format the kernels read (bfloat16 bit patterns, or OCP e4m3
codes with one per-tensor scale).

Recipe (numpy ``Generator(PCG64(seed))``):
  * draw float32 standard normals in the order Q [B,Hq,S,d], K [B,Hkv,S,d],
    V [B,Hkv,S,d];
  * sharp keys: for each (b, hkv) in order, ``round(0.02*S)`` positions from
    ``permutation(S)`` of the same generator; those K rows are multiplied by 4;
  * BF16: round to nearest even;
  * FP8: per-tensor scale s = amax|X| / 448 (fp32), code = e4m3 of X / s
    (round to nearest, ties to even code, saturate at 448); descale = s.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

BF16, FP8_E4M3 = 0, 1
E4M3_MAX = 448.0


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    S: int
    d: int
    causal: bool
    dtype: int
    sharp: bool
    seed: int

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))

    def flops(self) -> float:
        """Attention FLOPs in the FlashAttention convention."""
        full = 4.0 * self.B * self.Hq * self.S * self.S * self.d
        return full / 2.0 if self.causal else full

    def score_elements(self) -> float:
        if self.causal:
            return float(self.B * self.Hq) * self.S * (self.S + 1) / 2.0
        return float(self.B * self.Hq) * self.S * self.S


# The paper's timing shapes (App. B.3: batch 1, 16 heads, head dim 128, S up to
# 16K; GQA 32/8 in Table B4e) and a small shape the oracle finishes quickly.
WORKLOADS = {
    w.name: w
    for w in [
        Workload("noncausal_bf16_b1_h2_s256_d64", 1, 2, 2, 256, 64, False, BF16, False, 1000),
        Workload("causal_bf16_b4_h32kv8_s2048_d128_sharp", 4, 32, 8, 2048, 128, True, BF16, True, 1001),
        Workload("noncausal_fp8_b2_h16_s8192_d128", 2, 16, 16, 8192, 128, False, FP8_E4M3, False, 1002),
        Workload("causal_fp8_b2_h32kv8_s8192_d128_sharp", 2, 32, 8, 8192, 128, True, FP8_E4M3, True, 1003),
        Workload("causal_bf16_b1_h64kv8_s16384_d128_sharp", 1, 64, 8, 16384, 128, True, BF16, True, 1004),
        Workload("causal_fp8_b1_h64kv8_s16384_d128_sharp", 1, 64, 8, 16384, 128, True, FP8_E4M3, True, 1004),
    ]
}


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (no NaN inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_decode(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint32) << 16).view(np.float32)


def _e4m3_table() -> np.ndarray:
    codes = np.arange(0x7F, dtype=np.int64)  # 0x00 .. 0x7E: every non-negative finite code
    e = (codes >> 3) & 15
    m = codes & 7
    sub = m.astype(np.float64) / 8.0 * 2.0 ** -6
    nrm = (1.0 + m.astype(np.float64) / 8.0) * np.exp2(e.astype(np.float64) - 7.0)
    return np.where(e == 0, sub, nrm)


_E4M3_POS = _e4m3_table()


def e4m3_decode(c: np.ndarray) -> np.ndarray:
    c = np.asarray(c, dtype=np.uint8)
    mag = _E4M3_POS[np.minimum(c & 0x7F, 0x7E)]
    return np.where(c & 0x80, -mag, mag)


def e4m3_codes(x: np.ndarray) -> np.ndarray:
    """Nearest finite e4m3 code, ties to the even code, saturating at 448."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.minimum(np.searchsorted(_E4M3_POS, a, side="left"), 0x7E)
    lo = np.maximum(hi - 1, 0)
    dlo = a - _E4M3_POS[lo]
    dhi = _E4M3_POS[hi] - a
    take_hi = (dhi < dlo) | ((dhi == dlo) & (hi % 2 == 0))
    mag = np.where(take_hi, hi, lo).astype(np.uint8)
    return np.where(np.signbit(x), mag | 0x80, mag).astype(np.uint8)


def quantize_e4m3(x: np.ndarray) -> tuple[np.ndarray, float]:
    """Per-tensor e4m3 quantisation: (codes, descale)."""
    amax = np.float32(np.max(np.abs(x)))
    s = np.float32(amax / np.float32(E4M3_MAX)) if amax > 0 else np.float32(1.0)
    codes = e4m3_codes((np.asarray(x, np.float32) / s).astype(np.float32))
    return codes, float(s)


@dataclass
class Inputs:
    q: np.ndarray  # uint16 bf16 bits or uint8 e4m3 codes, [B,Hq,S,d]
    k: np.ndarray  # [B,Hkv,S,d]
    v: np.ndarray
    descale: tuple[float, float, float]
    dtype: int


def make_inputs(B: int, Hq: int, Hkv: int, S: int, d: int, dtype: int, sharp: bool,
                seed: int) -> Inputs:
    rng = np.random.Generator(np.random.PCG64(seed))
    q = rng.standard_normal((B, Hq, S, d), dtype=np.float32)
    k = rng.standard_normal((B, Hkv, S, d), dtype=np.float32)
    v = rng.standard_normal((B, Hkv, S, d), dtype=np.float32)
    if sharp:
        n_sharp = int(round(0.02 * S))
        for b in range(B):
            for h in range(Hkv):
                idx = rng.permutation(S)[:n_sharp]
                k[b, h, idx, :] *= np.float32(4.0)
    if dtype == BF16:
        return Inputs(bf16_bits(q), bf16_bits(k), bf16_bits(v), (1.0, 1.0, 1.0), BF16)
    qc, qs = quantize_e4m3(q)
    kc, ks = quantize_e4m3(k)
    vc, vs = quantize_e4m3(v)
    return Inputs(qc, kc, vc, (qs, ks, vs), FP8_E4M3)


def workload_inputs(w: Workload) -> Inputs:
    return make_inputs(w.B, w.Hq, w.Hkv, w.S, w.d, w.dtype, w.sharp, w.seed)


def make_decode_inputs(B: int, Hq: int, Hkv: int, Sq: int, Sk_cap: int, d: int, dtype: int, sharp: bool,
                       seed: int) -> Inputs:
    """Decode inputs: Q [B,Hq,Sq,d] and a key/value cache K, V [B,Hkv,Sk_cap,d],
    drawn and stored with the same recipe as make_inputs (sharp keys among the
    cache rows: round(0.02 * Sk_cap) per (b, hkv))."""
    rng = np.random.Generator(np.random.PCG64(seed))
    q = rng.standard_normal((B, Hq, Sq, d), dtype=np.float32)
    k = rng.standard_normal((B, Hkv, Sk_cap, d), dtype=np.float32)
    v = rng.standard_normal((B, Hkv, Sk_cap, d), dtype=np.float32)
    if sharp:
        n_sharp = int(round(0.02 * Sk_cap))
        for b in range(B):
            for h in range(Hkv):
                idx = rng.permutation(Sk_cap)[:n_sharp]
                k[b, h, idx, :] *= np.float32(4.0)
    if dtype == BF16:
        return Inputs(bf16_bits(q), bf16_bits(k), bf16_bits(v), (1.0, 1.0, 1.0), BF16)
    qc, qs = quantize_e4m3(q)
    kc, ks = quantize_e4m3(k)
    vc, vs = quantize_e4m3(v)
    return Inputs(qc, kc, vc, (qs, ks, vs), FP8_E4M3)
