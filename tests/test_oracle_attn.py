"""Pins of the oracle's attention modes.

EXACT is checked against torch's scaled_dot_product_attention in float64 on
the CPU (a library routine).  The Rowmax-H15 modes are checked against
special cases with closed forms (integer base-two logit differences reduce
H15 to exact softmax; uniform logits give uniform weights), a non-recurrent
prefix-max form of the per-tile recurrence evaluated in exact rationals,
brute force with Python fractions, and the invariants the paper states."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2609_33586_amd import synth

BF16, FP8 = oracle.BF16, oracle.FP8_E4M3


def dequant(inp: synth.Inputs):
    dec = synth.bf16_decode if inp.dtype == BF16 else synth.e4m3_decode
    qd, kd, vd = inp.descale
    return (np.asarray(dec(inp.q), np.float64) * qd, np.asarray(dec(inp.k), np.float64) * kd,
            np.asarray(dec(inp.v), np.float64) * vd)


def sdpa(inp: synth.Inputs, causal: bool, scale: float):
    q, k, v = (torch.from_numpy(x) for x in dequant(inp))
    g = q.shape[1] // k.shape[1]
    k = k.repeat_interleave(g, dim=1)
    v = v.repeat_interleave(g, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=causal, scale=scale)
    s = (q @ k.transpose(-1, -2)) * scale
    if causal:
        S = s.shape[-1]
        s = s.masked_fill(torch.triu(torch.ones(S, S, dtype=torch.bool), 1), float("-inf"))
    return o.numpy(), torch.logsumexp(s, dim=-1).numpy()


@pytest.mark.parametrize("dtype", [BF16, FP8])
@pytest.mark.parametrize("causal", [False, True])
def test_exact_mode_matches_sdpa(dtype, causal):
    inp = synth.make_inputs(2, 4, 2, 67, 16, dtype, sharp=True, seed=11)
    scale = 0.25
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=dtype, causal=causal, scale=scale,
                         mode=oracle.EXACT, descale=inp.descale)
    o_ref, lse_ref = sdpa(inp, causal, scale)
    assert np.max(np.abs(o - o_ref)) < 1e-12
    assert np.max(np.abs(lse - lse_ref)) < 1e-12


def test_exact_mode_row_subset_matches_full():
    inp = synth.make_inputs(1, 2, 1, 40, 8, BF16, sharp=False, seed=12)
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE, Bc=16)
    rows = np.array([79, 0, 41, 5])
    o2, lse2 = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE,
                           Bc=16, rows=rows)
    assert np.array_equal(o2, o.reshape(-1, 8)[rows]) and np.array_equal(lse2, lse.reshape(-1)[rows])


def integer_inputs(B, Hq, Hkv, S, d, rng, lo=-2, hi=2):
    """bf16 operands holding small integers, so every raw logit is an integer."""
    q = rng.integers(lo, hi + 1, (B, Hq, S, d)).astype(np.float32)
    k = rng.integers(lo, hi + 1, (B, Hkv, S, d)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, S, d)).astype(np.float32)
    return synth.Inputs(synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v), (1.0, 1.0, 1.0), BF16)


SCALE_C1_ONE = 1.0 / math.log2(math.e)  # c1 = fp32(scale * log2 e) = 1 exactly


@pytest.mark.parametrize("mode", [oracle.H15_TILE, oracle.H15_WHOLEROW])
@pytest.mark.parametrize("causal", [False, True])
def test_h15_equals_softmax_when_differences_are_whole_octaves(mode, causal):
    # With c1 = 1 and integer logits, 2x = 2(s - m) is an even integer, so
    # every H15 weight is exactly 2^(s - m): H15 attention = softmax attention.
    assert oracle.c1(SCALE_C1_ONE) == 1.0
    rng = np.random.default_rng(5)
    inp = integer_inputs(1, 4, 2, 45, 4, rng)
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=causal, scale=SCALE_C1_ONE, mode=mode, Bc=8)
    o_ref, lse_ref = sdpa(inp, causal, SCALE_C1_ONE)
    assert np.max(np.abs(o - o_ref)) < 1e-12
    assert np.max(np.abs(lse - lse_ref)) < 1e-12


def test_h15_fp8_offset_cancels_for_whole_octaves():
    # FP8 path: the offset 8 multiplies every weight by 2^8 and cancels.
    rng = np.random.default_rng(6)
    q = rng.integers(-1, 2, (1, 2, 32, 4)).astype(np.float32)
    k = rng.integers(-1, 2, (1, 2, 32, 4)).astype(np.float32)
    v = rng.integers(-3, 4, (1, 2, 32, 4)).astype(np.float32)
    inp = synth.Inputs(synth.e4m3_codes(q), synth.e4m3_codes(k), synth.e4m3_codes(v), (1.0, 1.0, 1.0), FP8)
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=FP8, causal=True, scale=SCALE_C1_ONE, mode=oracle.H15_TILE, Bc=8)
    o_ref, lse_ref = sdpa(inp, True, SCALE_C1_ONE)
    # logits lie in [-4, 4], so every P = e4m3(2^(8 + s - m)) >= 1 is exact
    assert np.max(np.abs(o - o_ref)) < 1e-12
    assert np.max(np.abs(lse - lse_ref)) < 1e-12


def test_h15_half_octave_ratio():
    # Half-integer base-two differences: odd n, weight 1.5 * 2^((n-1)/2)
    # against exact 2^(n/2), a ratio of 1.5/sqrt(2).
    s = np.array([0.0, -0.5, -1.5, -2.5, -1.0, -3.0], np.float32)
    w, p, _ = oracle.h15_row_from_logits(s, 0, False, 1.0, BF16, Bc=64)
    exact = 2.0 ** s.astype(np.float64)
    ratio = w / exact
    n = 2 * s
    # RNE of an odd integer n is n itself; even n gives ratio 1.
    for r, nn in zip(ratio, n):
        want = 1.5 / math.sqrt(2.0) if int(nn) % 2 else 1.0
        assert abs(r - want) < 1e-15


@pytest.mark.parametrize("dtype", [BF16, FP8])
@pytest.mark.parametrize("causal", [False, True])
def test_uniform_logits_give_uniform_weights(dtype, causal):
    rng = np.random.default_rng(7)
    S, d = 70, 8
    q = rng.standard_normal((1, 1, S, d)).astype(np.float32)
    krow = rng.standard_normal(d).astype(np.float32)
    k = np.broadcast_to(krow, (1, 1, S, d)).copy()
    v = rng.standard_normal((1, 1, S, d)).astype(np.float32)
    if dtype == BF16:
        inp = synth.Inputs(synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v), (1.0, 1.0, 1.0), BF16)
    else:
        inp = synth.Inputs(synth.e4m3_codes(q), synth.e4m3_codes(k), synth.e4m3_codes(v), (1.0, 1.0, 1.0), FP8)
    _, _, vdq = dequant(inp)
    for mode in (oracle.H15_TILE, oracle.H15_WHOLEROW, oracle.ROWMAX_POT):
        o, _ = oracle.attn(inp.q, inp.k, inp.v, dtype=dtype, causal=causal, scale=0.37, mode=mode, Bc=16)
        for i in range(S):
            n = i + 1 if causal else S
            assert np.max(np.abs(o[0, 0, i] - vdq[0, 0, :n].mean(axis=0))) < 1e-12
    # and the weight at every key is 2^off
    s = np.full(S, 1.25, np.float32)
    w, _, _ = oracle.h15_row_from_logits(s, S - 1, causal, 0.3, dtype, 16)
    assert np.all(w == (256.0 if dtype == FP8 else 1.0))


def test_causal_never_reads_future_values():
    rng = np.random.default_rng(8)
    inp = synth.make_inputs(1, 2, 2, 48, 8, BF16, sharp=False, seed=13)
    o, _ = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE, Bc=16)
    for i in (0, 15, 16, 30):
        v2 = inp.v.copy()
        v2[:, :, i + 1:, :] = synth.bf16_bits(np.full((1,), 1e30, np.float32))[0]
        o2, _ = oracle.attn(inp.q, inp.k, v2, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE, Bc=16)
        assert np.array_equal(o2[:, :, i], o[:, :, i])


def test_tile_at_least_s_equals_whole_row():
    inp = synth.make_inputs(1, 2, 1, 100, 16, BF16, sharp=True, seed=14)
    a, la = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.25, mode=oracle.H15_TILE, Bc=128)
    b, lb = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.25, mode=oracle.H15_WHOLEROW)
    assert np.array_equal(a, b) and np.array_equal(la, lb)
    # with a smaller tile the per-tile anchor differs somewhere
    c, _ = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.25, mode=oracle.H15_TILE, Bc=8)
    assert not np.array_equal(a, c)


# ---- exact-rational evaluation of the non-recurrent form ------------------

def round_f32(x: Fraction) -> np.float32:
    """Correctly rounded (nearest, ties to even) fp32 value of a rational."""
    f = np.float32(float(x))
    best = f
    for c in (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))):
        dc, db = abs(Fraction(float(c)) - x), abs(Fraction(float(best)) - x)
        if dc < db or (dc == db and (int(np.array([c]).view(np.uint32)[0]) & 1) == 0):
            best = c
    return best


def h15_fraction(y: Fraction) -> Fraction:
    """Eq. (m-h15) in exact arithmetic, input clamped at -252 (App. B.1)."""
    y = max(y, Fraction(-252))
    n = round(y)  # Python rounds a Fraction half to even
    return (1 + Fraction(n % 2, 2)) * Fraction(2) ** (n // 2)


def prefix_max_form(s: np.ndarray, v: np.ndarray, jend: int, c1: np.float32, Bc: int, off: int):
    """O and LSE of one row written without the online recurrence: key j,
    in tile t(j), is weighted by H15(y_j) relative to the prefix max M_t(j)
    of the tiles up to its own, times 2^(c1 (M_t(j) - M_final)) -- the
    product of every later rescale factor."""
    c2 = np.float32(2.0) * c1
    tiles = [(t0, min(t0 + Bc, jend)) for t0 in range(0, jend, Bc)]
    prefix = []
    m = -np.inf
    for t0, t1 in tiles:
        m = max(m, float(np.max(s[t0:t1])))
        prefix.append(np.float32(m))
    M = float(prefix[-1])
    num = np.zeros(v.shape[1])
    den = 0.0
    for (t0, t1), Mt in zip(tiles, prefix):
        nb = round_f32(-Fraction(float(Mt)) * Fraction(float(c2)) + 2 * off)
        for j in range(t0, t1):
            y = round_f32(Fraction(float(s[j])) * Fraction(float(c2)) + Fraction(float(nb)))
            w = float(h15_fraction(Fraction(float(y)))) * 2.0 ** (float(c1) * (float(Mt) - M))
            num += w * v[j]
            den += w
    return num / den, math.log(2) * (M * float(c1) + math.log2(den) - off)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Bc", [1, 7, 16, 1000])
def test_tile_recurrence_matches_prefix_max_form(causal, Bc):
    inp = synth.make_inputs(1, 2, 2, 53, 8, BF16, sharp=True, seed=15)
    scale = 0.9
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=causal, scale=scale, mode=oracle.H15_TILE, Bc=Bc)
    c1 = np.float32(oracle.c1(scale))
    _, _, vdq = dequant(inp)
    for h in range(2):
        for i in (0, 6, 7, 26, 52):
            s = oracle.logits_row(inp.q, inp.k, BF16, 0, h, i)
            jend = i + 1 if causal else 53
            o_ref, lse_ref = prefix_max_form(s, vdq[0, h], jend, c1, Bc, 0)
            assert np.max(np.abs(o[0, h, i] - o_ref)) < 1e-12
            assert abs(lse[0, h, i] - lse_ref) < 1e-12


def test_logits_are_exact_dot_products_rounded_once():
    inp = synth.make_inputs(1, 1, 1, 20, 16, BF16, sharp=True, seed=16)
    q, k, _ = dequant(inp)
    for i in (0, 19):
        s = oracle.logits_row(inp.q, inp.k, BF16, 0, 0, i)
        for j in range(20):
            exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(q[0, 0, i], k[0, 0, j]))
            assert s[j] == round_f32(exact)


def test_brute_force_tiny_with_fractions():
    # S=4, d=2, integer q/k, c1 = 1, tile 2: the tile recurrence by hand in
    # exact rationals, values v_j = j + 1.
    q = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0], [2.0, -1.0]], np.float32)
    k = np.array([[0.5, 0.0], [1.5, 1.0], [-1.0, 2.5], [3.0, 0.5]], np.float32)
    v = np.array([[1.0, -1.0], [2.0, 0.0], [3.0, 4.0], [4.0, 2.0]], np.float32)
    inp = synth.Inputs(synth.bf16_bits(q[None, None]), synth.bf16_bits(k[None, None]),
                       synth.bf16_bits(v[None, None]), (1.0, 1.0, 1.0), BF16)
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=False, scale=SCALE_C1_ONE, mode=oracle.H15_TILE, Bc=2)
    for i in range(4):
        s = [Fraction(float(q[i] @ k[j])) for j in range(4)]  # exact: halves times small integers
        m1 = max(s[0:2])
        w = [h15_fraction(2 * (s[j] - m1)) for j in range(2)]
        m2 = max(m1, max(s[2:4]))
        # rescale of tile 1 by 2^(m1 - m2): an integer or half-integer power of two
        alpha = 2.0 ** float(m1 - m2)
        w += [h15_fraction(2 * (s[j] - m2)) for j in range(2, 4)]
        num = [alpha * float(w[0] * Fraction(float(v[0, c])) + w[1] * Fraction(float(v[1, c])))
               + float(w[2] * Fraction(float(v[2, c])) + w[3] * Fraction(float(v[3, c]))) for c in range(2)]
        den = alpha * float(w[0] + w[1]) + float(w[2] + w[3])
        for c in range(2):
            assert abs(o[0, 0, i, c] - num[c] / den) < 1e-14
        assert abs(lse[0, 0, i] - math.log(2) * (float(m2) + math.log2(den))) < 1e-14


def test_anchor_weight_is_exactly_one_and_bounded():
    inp = synth.make_inputs(1, 1, 1, 300, 32, BF16, sharp=True, seed=17)
    for dtype, top in ((BF16, 1.0), (FP8, 256.0)):
        for i in (0, 99, 200, 299):
            s = oracle.logits_row(inp.q, inp.k, BF16, 0, 0, i)
            w, _, _ = oracle.h15_row_from_logits(s, i, True, 0.2, dtype, Bc=64)
            j = int(np.argmax(s[: i + 1]))
            assert w[j] == top
            assert np.all(w[: i + 1] <= top) and np.all(w[i + 1:] == 0)


def test_fp8_weights_are_bf16_weights_times_256():
    inp = synth.make_inputs(1, 1, 1, 200, 32, BF16, sharp=True, seed=18)
    for i in (10, 150):
        s = oracle.logits_row(inp.q, inp.k, BF16, 0, 0, i)
        w0, _, _ = oracle.h15_row_from_logits(s, i, False, 0.2, BF16, Bc=64)
        w8, _, _ = oracle.h15_row_from_logits(s, i, False, 0.2, FP8, Bc=64)
        nz = w0 >= 2.0 ** -118
        assert np.array_equal(w8[nz], w0[nz] * 256.0)


def test_normalized_ratio_within_paper_bound():
    # App. B.2: envelope [-0.25, 0.335] on the unnormalised weights implies
    # |log2(p_hat / p)| <= 0.585 after normalisation (whole-row anchor).
    inp = synth.make_inputs(1, 1, 1, 256, 64, BF16, sharp=True, seed=19)
    c1 = oracle.c1(0.125)
    for i in (0, 100, 255):
        s = oracle.logits_row(inp.q, inp.k, BF16, 0, 0, i)
        w, _, _ = oracle.h15_row_from_logits(s, i, False, c1, BF16, Bc=256)
        x = (s.astype(np.float64) - s.max()) * c1
        p = 2.0 ** x / np.sum(2.0 ** x)
        ph = w / w.sum()
        r = np.log2(ph / p)
        assert np.max(np.abs(r)) <= 0.585 + 1e-4


def test_rowmax_pot_closed_forms():
    # Eq. (rowmax-pot): d_j = min(20, floor(x_j + 1/2)), x_j = Delta_j / ln 2.
    q = np.array([[[[1.0, 0.0]]]], np.float32)
    k = np.array([[[[0.0, 0.0], [-1.0, 0.0], [-2.5, 0.0], [-25.0, 0.0], [-3.25, 0.0]]]], np.float32)
    qq = np.repeat(q, 5, axis=2)
    v = np.eye(5, 2, dtype=np.float32)[None, None] * 0 + np.arange(5, dtype=np.float32)[None, None, :, None]
    inp = synth.Inputs(synth.bf16_bits(qq), synth.bf16_bits(k), synth.bf16_bits(v), (1.0, 1.0, 1.0), BF16)
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=False, scale=math.log(2), mode=oracle.ROWMAX_POT)
    # scale ln 2: Delta_j = ln2 * (0 - s_j), x_j = -s_j = 0, 1, 2.5, 25, 3.25
    d = np.array([0, 1, 3, 20, 3])  # floor(2.5 + .5) = 3 (half rounds up); 25 clamps to 20
    w = 2.0 ** -d
    assert abs(o[0, 0, 0, 0] - np.sum(w * np.arange(5)) / w.sum()) < 1e-14
    assert abs(lse[0, 0, 0] - math.log(w.sum())) < 1e-14


def test_exact_tile_close_to_exact():
    inp = synth.make_inputs(1, 2, 2, 96, 32, BF16, sharp=True, seed=20)
    a, _ = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.18, mode=oracle.EXACT)
    b, _ = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.18, mode=oracle.EXACT_TILE, Bc=32)
    vmax = np.max(np.abs(synth.bf16_decode(inp.v)))
    assert np.max(np.abs(a - b)) < 2.0 ** -8 * vmax


def test_rowmax_pot_row_from_logits_closed_forms():
    # the kernel-arithmetic form of Eq. (rowmax-pot): c1 = 1 makes x_j = m - s_j
    s = np.array([0.0, -1.0, -2.5, -25.0, -3.25, -0.5, -1.5, -19.5, -19.49], np.float32)
    w, p, lse = oracle.pot_row_from_logits(s, 8, False, 1.0)
    d = np.array([0, 1, 3, 20, 3, 1, 2, 20, 19])  # half rounds up; the tail clamps at 20
    assert np.array_equal(w, (2.0 ** -d).astype(np.float32))
    assert np.array_equal(p, np.array([int(np.array([x], np.float32).view(np.uint32)[0]) >> 16 for x in w]))
    assert abs(lse - math.log(2) * math.log2(np.sum(2.0 ** -d))) < 1e-14
    # causal: keys after the row carry nothing, and the anchor is the row's own max
    w, p, _ = oracle.pot_row_from_logits(np.array([-1.0, -3.0, 5.0], np.float32), 1, True, 1.0)
    assert list(w) == [1.0, 0.25, 0.0] and p[2] == 0
    # a shift of every logit by an exactly representable constant changes nothing
    w2, _, _ = oracle.pot_row_from_logits(s + np.float32(64.0), 8, False, 1.0)
    assert np.array_equal(w2, oracle.pot_row_from_logits(s, 8, False, 1.0)[0])


def test_rowmax_pot_row_form_matches_fp64_operator():
    # integer logits and c1 = 1: every gap is exact in both arithmetics, so
    # the row form's weights give the fp64 operator's O and LSE
    rng = np.random.default_rng(41)
    inp = integer_inputs(1, 2, 1, 40, 4, rng, lo=-3, hi=3)
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=SCALE_C1_ONE, mode=oracle.ROWMAX_POT)
    _, _, vdq = dequant(inp)
    for h in range(2):
        for i in (0, 9, 39):
            s = oracle.logits_row(inp.q, inp.k, BF16, 0, h, i)
            w, _, lse_row = oracle.pot_row_from_logits(s, i, True, 1.0)
            w = w.astype(np.float64)
            assert np.max(np.abs(o[0, h, i] - (w @ vdq[0, 0]) / w.sum())) < 1e-12
            assert abs(lse[0, h, i] - lse_row) < 1e-12


def exact_tile_prefix_form(s, v, jend, c1, Bc, off, dtype):
    """The exact-exp2 tile loop written out (diagnostic mode EXACT_TILE): key
    j in tile t gets W = fp32(2^y), y = fp32(s_j c1 + fp32(-M_t c1 + off)) with
    M_t the prefix max; PV uses W stored in the operand type (bf16 RNE or e4m3),
    the row sum W itself; every later rescale is 2^(c1 (M_t - M))."""
    tiles = [(t0, min(t0 + Bc, jend)) for t0 in range(0, jend, Bc)]
    m, prefix = -np.inf, []
    for t0, t1 in tiles:
        m = max(m, float(np.max(s[t0:t1])))
        prefix.append(np.float32(m))
    M = float(prefix[-1])
    num = np.zeros(v.shape[1])
    den = 0.0
    for (t0, t1), Mt in zip(tiles, prefix):
        nb = round_f32(-Fraction(float(Mt)) * Fraction(float(c1)) + off)
        for j in range(t0, t1):
            y = round_f32(Fraction(float(s[j])) * Fraction(float(c1)) + Fraction(float(nb)))
            w = np.float32(2.0 ** float(y))
            if dtype == BF16:
                pv = float(synth.bf16_decode(synth.bf16_bits(np.array([w], np.float32)))[0])
            else:
                pv = float(synth.e4m3_decode(synth.e4m3_codes(np.array([w], np.float64)))[0])
            f = 2.0 ** (float(c1) * (float(Mt) - M))
            num += pv * f * v[j]
            den += float(w) * f
    return num / den, math.log(2) * (M * float(c1) + math.log2(den) - off)


@pytest.mark.parametrize("dtype", [BF16, FP8])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("Bc", [1, 16, 1000])
def test_exact_tile_matches_prefix_max_form(dtype, causal, Bc):
    inp = synth.make_inputs(1, 2, 2, 53, 8, dtype, sharp=True, seed=21)
    scale = 0.7
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=dtype, causal=causal, scale=scale, mode=oracle.EXACT_TILE,
                         descale=(1.0, 1.0, 1.0), Bc=Bc)
    c1 = np.float32(oracle.c1(scale))
    off = 8 if dtype == FP8 else 0
    vdec = (synth.bf16_decode(inp.v) if dtype == BF16 else synth.e4m3_decode(inp.v)).astype(np.float64)
    for h in range(2):
        for i in (0, 7, 26, 52):
            s = oracle.logits_row(inp.q, inp.k, dtype, 0, h, i)
            jend = i + 1 if causal else 53
            o_ref, lse_ref = exact_tile_prefix_form(s, vdec[0, h], jend, c1, Bc, off, dtype)
            # the only step not fixed to the bit is the fp64 exp2 before its
            # fp32 rounding (libm's exp2 here, pow in the form above)
            assert np.max(np.abs(o[0, h, i] - o_ref)) < 1e-9 * np.max(np.abs(vdec))
            assert abs(lse[0, h, i] - lse_ref) < 1e-9


@pytest.mark.parametrize("k,mode", [(1, oracle.H15_TILE), (2, oracle.SQ4_TILE), (3, oracle.SQ8_TILE)])
@pytest.mark.parametrize("causal", [False, True])
def test_row_exponents_reproduce_the_weights(k, mode, causal):
    # y[j] = fp32(s_j ck + fp32(-M_t ck + 2^k off)) with M_t the prefix max of
    # key j's tile (anchor[j]); the weight realisation applied to y gives W.
    inp = synth.make_inputs(1, 1, 1, 90, 16, FP8, sharp=True, seed=22)
    sc = 0.2
    c1 = np.float32(oracle.c1(sc, inp.descale[0], inp.descale[1]))
    Bc = 32
    for i in (5, 40, 89):
        s = oracle.logits_row(inp.q, inp.k, FP8, 0, 0, i)
        y, anchor, w = oracle.row_exponents_from_logits(s, i, causal, float(c1), FP8, Bc, k=k)
        w2, _, _ = oracle.sq_row_from_logits(s, i, causal, float(c1), FP8, Bc, k=k)
        assert np.array_equal(w.view(np.uint32), w2.view(np.uint32))
        jend = i + 1 if causal else 90
        assert np.all(np.isneginf(y[jend:])) and np.all(np.isneginf(anchor[jend:]))
        ck = Fraction(float(c1)) * 2 ** k
        m = -np.inf
        for j in range(jend):
            if j % Bc == 0:
                m = max(m, float(np.max(s[j:min(j + Bc, jend)])))
            assert anchor[j] == np.float32(m)
            nb = round_f32(-Fraction(m) * ck + 2 ** k * 8)
            assert y[j] == round_f32(Fraction(float(s[j])) * ck + Fraction(float(nb)))
            assert w[j] == np.float32(oracle.sq_weight(float(y[j]), k))
