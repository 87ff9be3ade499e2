"""The kernel's 16-bit lane finishing of the lattice weights, restated on the
CPU and checked against the oracle's weights (App. B.1 "Implementation",
App. B.2 ablation).

A lattice weight S(Q_{2^-k}(x)) with k <= 3 has at most k mantissa bits, so
the low half of its FP32 pattern is zero and the top half is its BF16
pattern.  The kernel packs two keys per register and finishes them in 16-bit
lanes: the lane holds the low half of bits(t) with t = y + 0x4B400000
(RNE(y) modulo 2^16, the magic's low half being zero), is clamped at
-126 * 2^k as int16 when every |y| < 2^15 (the narrow mode) or was clamped
in FP32 before the add, and becomes lane * 2^(7-k) + 0x3F80 modulo 2^16.
Masked keys enter with the lane value 385 * 2^k, whose result is +0.

These tests emulate that integer recipe with numpy (no GPU) and require the
oracle's bits for every rounded exponent the narrow mode can meet, ties
included, and for random FP32 exponents across the FP32-clamp range."""
import numpy as np
import pytest

import oracle

MAGIC = np.float32(12582912.0)  # 0x4B400000


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def lane_finish(lane16, k):
    """lane * 2^(7-k) + 0x3F80 modulo 2^16 (the packed multiply-add)."""
    return (lane16.astype(np.uint32) * (1 << (7 - k)) + 0x3F80) & 0xFFFF


def narrow_recipe(y, k):
    t = (np.asarray(y, np.float32) + MAGIC).astype(np.float32)
    lane = (bits(t) & 0xFFFF).astype(np.uint16).view(np.int16)
    lane = np.maximum(lane, np.int16(-126 * (1 << k)))
    return lane_finish(lane.view(np.uint16), k)


def fp32_clamp_recipe(y, k):
    yc = np.maximum(np.asarray(y, np.float32), np.float32(-126.0 * (1 << k)))
    t = (yc + MAGIC).astype(np.float32)
    return lane_finish((bits(t) & 0xFFFF).astype(np.uint16), k)


def oracle_top_halves(y, k):
    w = np.array([oracle.sq_weight(float(v), k) for v in y], np.float32)
    wb = bits(w)
    # every lattice weight is a BF16 value: the low half is zero
    assert np.all((wb & 0xFFFF) == 0)
    return wb >> 16


def narrow_grid(k):
    """Every integer in the narrow range, the ties between them, and points
    a quarter away, as fp32."""
    hi = 8 * (1 << k)
    n = np.arange(-32767, hi + 1, dtype=np.float64)
    return np.unique(np.concatenate([n, n + 0.5, n + 0.25, n - 0.25]).astype(np.float32))


@pytest.mark.parametrize("k", [1, 2, 3])
def test_narrow_lane_clamp_matches_oracle(k):
    y = narrow_grid(k)
    y = y[np.abs(y) < 32767]
    want = oracle_top_halves(y, k)
    got = narrow_recipe(y, k)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"k={k}: {bad.size} mismatches, first y={y[bad[0]]}"


@pytest.mark.parametrize("k", [1, 2, 3])
def test_fp32_clamp_lane_finish_matches_oracle(k):
    rng = np.random.default_rng(300 + k)
    y = np.concatenate([
        -rng.uniform(0, 2.0 ** 22, 20000), -rng.uniform(0, 300 * (1 << k), 20000),
        rng.uniform(0, 8 * (1 << k), 2000), np.arange(-130 * (1 << k), 8 * (1 << k) + 1) + 0.5,
    ]).astype(np.float32)
    want = oracle_top_halves(y, k)
    got = fp32_clamp_recipe(y, k)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"k={k}: {bad.size} mismatches, first y={y[bad[0]]}"


@pytest.mark.parametrize("k", [1, 2, 3])
def test_masked_lane_value_gives_plus_zero(k):
    m = 385 * (1 << k)
    # above the narrow clamp, inside int16, and finished to +0
    assert -126 * (1 << k) <= m < 2 ** 15
    assert lane_finish(np.array([m], np.uint16), k)[0] == 0


def test_narrow_mode_does_not_cover_wrapped_lanes():
    # Outside |y| < 2^15 the low half no longer holds RNE(y) as an int16,
    # which is why the launcher falls back to the FP32 clamp there.
    y = np.array([-40000.0], np.float32)
    assert narrow_recipe(y, 1)[0] != oracle_top_halves(y, 1)[0]
