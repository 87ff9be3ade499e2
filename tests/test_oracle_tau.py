"""Pins of the oracle's conditional-rescale anchor rule (App. B.2,
"Conditional rescaling moves the anchor" and "Semantic simulation"): the
running max moves to max(m, mt) only when it grows by more than tau in
base-two units, decided per row (the paper's simulation) or shared by an
aligned group of 32 rows (FlashAttention-4's per-warp decision).  Checked
against closed forms in exact rationals, hand-built cases, the exactness of
the exponential under any anchor, and invariants."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2609_33586_amd import synth
from test_oracle_attn import SCALE_C1_ONE, dequant, round_f32, sdpa
from test_oracle_sq import sq_fraction

BF16, FP8 = oracle.BF16, oracle.FP8_E4M3
TILED = [(oracle.H15_TILE, 1), (oracle.SQ4_TILE, 2), (oracle.SQ8_TILE, 3)]


@pytest.mark.parametrize("mode,k", TILED)
@pytest.mark.parametrize("causal", [False, True])
def test_tau_zero_group_decision_equals_per_row(mode, k, causal):
    # with tau = 0 a row whose max did not grow keeps m = max(m, mt) anyway,
    # so sharing the decision changes nothing
    inp = synth.make_inputs(1, 2, 1, 150, 16, BF16, sharp=True, seed=31)
    a = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=causal, scale=0.4, mode=mode, Bc=16, tau=0.0)
    b = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=causal, scale=0.4, mode=mode, Bc=16, tau=0.0,
                    tau_group=32)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def frozen_anchor_form(s, v, jend, c1, Bc, off, k):
    """O and LSE when the anchor never moves after the first tile: every key
    is weighted relative to the first tile's max M0, with no rescale."""
    M0 = np.float32(np.max(s[:min(Bc, jend)]))
    ck = np.float32(2.0 ** k) * c1
    nb = round_f32(-Fraction(float(M0)) * Fraction(float(ck)) + 2 ** k * off)
    num, den = np.zeros(v.shape[1]), Fraction(0)
    for j in range(jend):
        y = round_f32(Fraction(float(s[j])) * Fraction(float(ck)) + Fraction(float(nb)))
        w = sq_fraction(Fraction(float(y)), k)
        num += float(w) * v[j]
        den += w
    return num / float(den), math.log(2) * (float(M0) * float(c1) + math.log2(float(den)) - off)


@pytest.mark.parametrize("mode,k", TILED)
@pytest.mark.parametrize("group", [1, 32])
def test_infinite_tau_freezes_the_first_anchor(mode, k, group):
    # logits in a narrow range so the frozen-anchor weights stay far from the clamp
    rng = np.random.default_rng(32)
    S, d = 90, 8
    q = (rng.standard_normal((1, 1, S, d)) * 0.3).astype(np.float32)
    kk = (rng.standard_normal((1, 1, S, d)) * 0.3).astype(np.float32)
    v = rng.standard_normal((1, 1, S, d)).astype(np.float32)
    inp = synth.Inputs(synth.bf16_bits(q), synth.bf16_bits(kk), synth.bf16_bits(v), (1.0, 1.0, 1.0), BF16)
    scale = 0.8
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=False, scale=scale, mode=mode, Bc=16, tau=1e30,
                         tau_group=group)
    c1 = np.float32(oracle.c1(scale))
    _, _, vdq = dequant(inp)
    for i in (0, 17, 60, 89):
        s = oracle.logits_row(inp.q, inp.k, BF16, 0, 0, i)
        o_ref, lse_ref = frozen_anchor_form(s, vdq[0, 0], S, c1, 16, 0, k)
        assert np.max(np.abs(o[0, 0, i] - o_ref)) < 1e-12
        assert abs(lse[0, 0, i] - lse_ref) < 1e-12


def test_growth_by_exactly_tau_keeps_the_anchor():
    # c1 = 1, tiles of 2 keys, tau = 1.  Row logits: tile 0 max 0; tile 1 max
    # 1 (growth 1, not > 1: anchor stays 0, weight 2^1 = 2); tile 2 max 3
    # (growth 3 > 1: anchor moves to 3, earlier weights rescaled by 2^-3).
    s = np.array([0.0, -1.0, 1.0, 0.0, 3.0, 2.0], np.float32)
    w, p, lse = oracle.sq_row_from_logits(s, 5, False, 1.0, BF16, 2, k=1, tau=1.0)
    assert list(w) == [1.0, 0.5, 2.0, 1.0, 1.0, 0.5]
    # the weights are relative to the anchor of their own tile: l counts
    # (1 + 0.5 + 2 + 1) * 2^-3 + 1 + 0.5 and LSE = ln 2 (3 + log2 l)
    l = (1 + 0.5 + 2 + 1) * 2.0 ** -3 + 1.5
    assert abs(lse - math.log(2) * (3 + math.log2(l))) < 1e-14
    # with tau = 0 the anchor follows every growth
    w0, _, _ = oracle.sq_row_from_logits(s, 5, False, 1.0, BF16, 2, k=1, tau=0.0)
    assert list(w0) == [1.0, 0.5, 1.0, 0.5, 1.0, 0.5]


def test_group_decision_moves_every_row():
    # two rows, c1 = 1, tiles of 2, tau = 1: row 0 grows by 2 in tile 1 (moves),
    # row 1 grows by 0.5 (alone it would keep its anchor); shared, both move.
    s = np.array([[0.0, -1.0, 2.0, 1.0],
                  [0.0, -2.0, 0.5, -1.0]], np.float32)
    move = oracle.group_moves_from_logits(s, 0, False, 1.0, 2, 1.0)
    assert list(move[:2]) == [1, 1]
    w_alone, _, _ = oracle.sq_row_from_logits(s[1], 1, False, 1.0, BF16, 2, k=1, tau=1.0)
    w_group, _, _ = oracle.sq_row_from_logits_moves(s[1], 1, False, 1.0, BF16, 2, 1, move)
    # alone: anchor 0 for both tiles; shared: anchor 0.5 in tile 1
    assert w_alone[2] == oracle.h15_weight(2 * 0.5) and w_alone[3] == oracle.h15_weight(2 * -1.0)
    assert w_group[2] == 1.0 and w_group[3] == oracle.h15_weight(2 * -1.5)
    # and no row grew by more than 1 in a later tile: nothing moves
    s2 = np.array([[0.0, 0.0, 0.5, 0.0], [0.0, 0.0, 1.0, 0.0]], np.float32)
    assert list(oracle.group_moves_from_logits(s2, 0, False, 1.0, 2, 1.0)[:2]) == [1, 0]


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("group", [1, 32])
def test_exact_exponential_is_anchor_free(causal, group):
    # App. B.2: with an exact exponential the anchor does not matter, so the
    # conditional rescale gives back the exact denominator; only the bf16
    # storage of P remains (2^-9 relative)
    inp = synth.make_inputs(1, 2, 1, 200, 16, BF16, sharp=True, seed=33)
    sc = 0.3
    o, lse = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=causal, scale=sc, mode=oracle.EXACT_TILE, Bc=16,
                         tau=8.0, tau_group=group)
    o_ref, lse_ref = sdpa(inp, causal, sc)
    _, _, vdq = dequant(inp)
    assert np.max(np.abs(o - o_ref)) <= 2.0 ** -8 * np.max(np.abs(vdq))
    assert np.max(np.abs(lse - lse_ref)) < 1e-6


@pytest.mark.parametrize("mode,k", TILED)
def test_lagging_anchor_bounds_the_weights(mode, k):
    # with the anchor lagging by at most tau octaves, x <= tau and every
    # weight is at most 2^tau times the lattice's largest step above 2^x
    s = np.sort(np.random.default_rng(34).uniform(-3.0, 3.0, 300)).astype(np.float32)  # rising maxima
    tau = 8.0
    w, _, _ = oracle.sq_row_from_logits(s, 299, False, 1.3, BF16, 16, k=k, tau=tau)
    assert np.max(w) <= 2.0 ** (tau + 2.0 ** -k) and np.max(w) > 1.0
