"""Pins of the oracle's decode over a key/value cache (Sq query rows against
Sk cached keys, bottom-right causal alignment, the keys cut into parts that
each run the per-tile recurrence of App. B.1 / B.2 and merge exactly).

The paper leaves decode outside its scope, so these pins tie the decode form
to what is pinned already: with one part it is the square recurrence of the
same rows (bit for bit), the causal limit is the square mask shifted to the
cache's end, whole-octave logits reduce every cut to exact softmax, the part
semantics and the merge are evaluated independently in exact rationals, and
cache rows beyond Sk are never read."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2609_33586_amd import synth

BF16, FP8 = oracle.BF16, oracle.FP8_E4M3
TILED = (oracle.H15_TILE, oracle.SQ4_TILE, oracle.SQ8_TILE, oracle.EXACT_TILE)
SCALE_C1_ONE = 1.0 / math.log2(math.e)  # c1 = fp32(scale * log2 e) = 1 exactly


def square_with_tail(inp_dec, inp_sq, Sq, seed):
    """A square problem (Sk query rows) whose last Sq query rows are the
    decode queries: decode row i is square row Sk - Sq + i."""
    B, Hq, _, d = inp_dec.q.shape
    Sk = inp_sq.k.shape[2]
    qsq = np.array(inp_sq.q)
    qsq[:, :, Sk - Sq:, :] = inp_dec.q
    return synth.Inputs(qsq, inp_sq.k, inp_sq.v, inp_sq.descale, inp_sq.dtype)


@pytest.mark.parametrize("dtype", [BF16, FP8])
@pytest.mark.parametrize("mode", (oracle.EXACT,) + TILED)
@pytest.mark.parametrize("causal", [False, True])
def test_one_part_equals_square_rows(dtype, mode, causal):
    # Sq = 5 decode rows against Sk = 300 keys, one part: decode row i is the
    # square problem's row Sk - Sq + i (causal: its mask ends at that row),
    # bit for bit, for every mode.
    B, Hq, Hkv, Sk, Sq, d = 1, 4, 2, 300, 5, 16
    sq = synth.make_inputs(B, Hq, Hkv, Sk, d, dtype, sharp=True, seed=60)
    dec = synth.make_inputs(B, Hq, Hkv, Sq, d, dtype, sharp=False, seed=61)
    dec = synth.Inputs(dec.q, sq.k, sq.v, sq.descale, dtype)
    full = square_with_tail(dec, sq, Sq, 62)
    sc = 0.3
    o_d, l_d = oracle.decode(dec.q, dec.k, dec.v, Sk=Sk, dtype=dtype, causal=causal, scale=sc, mode=mode,
                             split_keys=0, descale=sq.descale, Bc=32)
    rows = np.array([(b * Hq + h) * Sk + Sk - Sq + i for b in range(B) for h in range(Hq) for i in range(Sq)])
    o_s, l_s = oracle.attn(full.q, full.k, full.v, dtype=dtype, causal=causal, scale=sc, mode=mode,
                           descale=sq.descale, Bc=32, rows=rows)
    assert np.array_equal(o_d.reshape(-1, d), o_s) and np.array_equal(l_d.reshape(-1), l_s)


@pytest.mark.parametrize("mode", (oracle.EXACT, oracle.H15_TILE))
def test_square_decode_is_square_causal(mode):
    # Sq = Sk: bottom-right alignment is the square causal mask itself
    inp = synth.make_inputs(1, 2, 1, 70, 8, BF16, sharp=True, seed=63)
    a, la = oracle.decode(inp.q, inp.k, inp.v, Sk=70, dtype=BF16, causal=True, scale=0.4, mode=mode,
                          split_keys=0, Bc=16)
    b, lb = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=True, scale=0.4, mode=mode, Bc=16)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_cache_rows_beyond_sk_are_never_read():
    Sk, cap = 150, 200
    inp = synth.make_inputs(1, 2, 1, cap, 16, BF16, sharp=True, seed=64)
    qd = synth.make_inputs(1, 2, 1, 3, 16, BF16, sharp=False, seed=65).q
    k2, v2 = np.array(inp.k), np.array(inp.v)
    k2[:, :, Sk:] = synth.bf16_bits(np.full((1, 1, cap - Sk, 16), 1e30, np.float32))
    v2[:, :, Sk:] = 0x7FC0  # NaN
    for mode in (oracle.EXACT, oracle.H15_TILE):
        for causal in (False, True):
            a, la = oracle.decode(qd, inp.k[:, :, :Sk], inp.v[:, :, :Sk], Sk=Sk, dtype=BF16, causal=causal,
                                  scale=0.25, mode=mode, split_keys=64, Bc=32)
            b, lb = oracle.decode(qd, k2, v2, Sk=Sk, dtype=BF16, causal=causal, scale=0.25, mode=mode,
                                  split_keys=64, Bc=32)
            assert np.array_equal(a, b) and np.array_equal(la, lb)


def test_split_at_least_sk_is_one_part_and_exact_ignores_parts():
    inp = synth.make_inputs(1, 4, 2, 260, 16, BF16, sharp=True, seed=66)
    qd = synth.make_inputs(1, 4, 2, 4, 16, BF16, sharp=True, seed=67).q
    kw = dict(Sk=260, dtype=BF16, causal=True, scale=0.35, Bc=32)
    a = oracle.decode(qd, inp.k, inp.v, mode=oracle.H15_TILE, split_keys=0, **kw)
    b = oracle.decode(qd, inp.k, inp.v, mode=oracle.H15_TILE, split_keys=288, **kw)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    # cutting the keys changes H15's anchors somewhere ...
    c = oracle.decode(qd, inp.k, inp.v, mode=oracle.H15_TILE, split_keys=64, **kw)
    assert not np.array_equal(a[0], c[0])
    # ... but not exact softmax
    e0 = oracle.decode(qd, inp.k, inp.v, mode=oracle.EXACT, split_keys=0, **kw)
    e1 = oracle.decode(qd, inp.k, inp.v, mode=oracle.EXACT, split_keys=64, **kw)
    assert np.array_equal(e0[0], e1[0]) and np.array_equal(e0[1], e1[1])


@pytest.mark.parametrize("split", [0, 16, 32, 96])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("mode", [oracle.H15_TILE, oracle.SQ4_TILE, oracle.SQ8_TILE])
def test_whole_octave_logits_reduce_every_cut_to_softmax(split, causal, mode):
    # c1 = 1 and integer logits: every lattice weight is exactly 2^(s - m)
    # whatever the anchor, so the parts, their merge factors 2^(m_p - m) and
    # the final normalisation must give exact softmax attention.
    rng = np.random.default_rng(68)
    B, Hq, Hkv, Sk, Sq, d = 1, 2, 1, 130, 3, 4
    q = rng.integers(-2, 3, (B, Hq, Sq, d)).astype(np.float32)
    k = rng.integers(-2, 3, (B, Hkv, Sk, d)).astype(np.float32)
    v = rng.standard_normal((B, Hkv, Sk, d)).astype(np.float32)
    qb, kb, vb = synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v)
    assert oracle.c1(SCALE_C1_ONE) == 1.0
    o, lse = oracle.decode(qb, kb, vb, Sk=Sk, dtype=BF16, causal=causal, scale=SCALE_C1_ONE, mode=mode,
                           split_keys=split, Bc=16)
    qd, kd, vd = (synth.bf16_decode(x).astype(np.float64) for x in (qb, kb, vb))
    for h in range(Hq):
        for i in range(Sq):
            jend = Sk - Sq + i + 1 if causal else Sk
            s = kd[0, 0, :jend] @ qd[0, h, i]
            w = 2.0 ** (s - s.max())
            assert np.max(np.abs(o[0, h, i] - (w @ vd[0, 0, :jend]) / w.sum())) < 1e-12
            assert abs(lse[0, h, i] - (s.max() * math.log(2) + math.log(w.sum()))) < 1e-12


def round_f32(x: Fraction) -> np.float32:
    f = np.float32(float(x))
    best = f
    for c in (np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))):
        dc, db = abs(Fraction(float(c)) - x), abs(Fraction(float(best)) - x)
        if dc < db or (dc == db and (int(np.array([c]).view(np.uint32)[0]) & 1) == 0):
            best = c
    return best


def h15_fraction(y: Fraction) -> Fraction:
    y = max(y, Fraction(-252))
    n = round(y)  # half to even
    return (1 + Fraction(n % 2, 2)) * Fraction(2) ** (n // 2)


def parts_form(s, v, jend, c1, Bc, split):
    """Decode O and LSE of one row written out part by part: key j of part p
    and tile t is weighted by H15 relative to the prefix max of the part's
    tiles up to t, times 2^(c1 (M_pt - M)) with M the row's overall max --
    every rescale inside the part and the part's merge factor in one."""
    Sk = len(s)
    part = Sk if split == 0 else split
    c2 = np.float32(2.0) * c1
    M = float(np.max(s[:jend]))
    num = np.zeros(v.shape[1])
    den = 0.0
    for j0 in range(0, min(Sk, jend), part):
        m = -np.inf
        for t0 in range(j0, min(j0 + part, jend), Bc):
            t1 = min(t0 + Bc, j0 + part, jend)
            m = max(m, float(np.max(s[t0:t1])))
            Mt = np.float32(m)
            nb = round_f32(-Fraction(float(Mt)) * Fraction(float(c2)))
            for j in range(t0, t1):
                y = round_f32(Fraction(float(s[j])) * Fraction(float(c2)) + Fraction(float(nb)))
                w = float(h15_fraction(Fraction(float(y)))) * 2.0 ** (float(c1) * (float(Mt) - M))
                num += w * v[j]
                den += w
    return num / den, math.log(2) * (M * float(c1) + math.log2(den))


@pytest.mark.parametrize("split", [0, 8, 24, 40])
@pytest.mark.parametrize("causal", [False, True])
def test_parts_match_the_written_out_form(split, causal):
    Sk, Sq, d, Bc = 61, 4, 8, 8
    inp = synth.make_inputs(1, 2, 2, Sk, d, BF16, sharp=True, seed=69)
    qd = synth.make_inputs(1, 2, 2, Sq, d, BF16, sharp=True, seed=70).q
    sc = 0.8
    o, lse = oracle.decode(qd, inp.k, inp.v, Sk=Sk, dtype=BF16, causal=causal, scale=sc, mode=oracle.H15_TILE,
                           split_keys=split, Bc=Bc)
    c1 = np.float32(oracle.c1(sc))
    vdq = synth.bf16_decode(inp.v).astype(np.float64)
    for h in range(2):
        for i in range(Sq):
            s = oracle.decode_logits_row(qd, inp.k, BF16, Sk, 0, h, i)
            jend = Sk - Sq + i + 1 if causal else Sk
            o_ref, lse_ref = parts_form(s, vdq[0, h], jend, c1, Bc, split)
            assert np.max(np.abs(o[0, h, i] - o_ref)) < 1e-12
            assert abs(lse[0, h, i] - lse_ref) < 1e-12


def test_decode_logits_are_exact_dot_products_rounded_once():
    inp = synth.make_inputs(1, 2, 1, 30, 16, FP8, sharp=True, seed=71)
    qd = synth.make_inputs(1, 2, 1, 2, 16, FP8, sharp=True, seed=72).q
    qv, kv = synth.e4m3_decode(qd), synth.e4m3_decode(inp.k)
    for h, i in ((0, 0), (1, 1)):
        s = oracle.decode_logits_row(qd, inp.k, FP8, 30, 0, h, i)
        for j in range(30):
            exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(qv[0, h, i], kv[0, 0, j]))
            assert s[j] == round_f32(exact)


@pytest.mark.parametrize("dtype", [BF16, FP8])
@pytest.mark.parametrize("split", [0, 64])
def test_row_from_logits_agrees_with_decode(dtype, split):
    Sk, Sq, d = 200, 3, 16
    inp = synth.make_inputs(1, 2, 1, Sk, d, dtype, sharp=True, seed=73)
    qd = synth.make_inputs(1, 2, 1, Sq, d, dtype, sharp=True, seed=74).q
    sc = 0.3
    _, lse = oracle.decode(qd, inp.k, inp.v, Sk=Sk, dtype=dtype, causal=True, scale=sc, mode=oracle.H15_TILE,
                           split_keys=split, descale=inp.descale, Bc=32)
    c1 = oracle.c1(sc, inp.descale[0], inp.descale[1])
    for i in range(Sq):
        s = oracle.decode_logits_row(qd, inp.k, dtype, Sk, 0, 1, i)
        jend = Sk - Sq + i + 1
        w, p, l_row = oracle.decode_row_from_logits(s, jend, c1, dtype, 32, split)
        assert abs(l_row - lse[0, 1, i]) < 1e-12
        assert np.all(w[jend:] == 0) and np.all(p[jend:] == 0) and np.all(w[:jend] > 0)
        # every weight of a part is relative to the part's own running max:
        # the first key of every part's first tile that holds its max gets 2^off
        off = 8 if dtype == FP8 else 0
        part = Sk if split == 0 else split
        for j0 in range(0, jend, part):
            t1 = min(j0 + 32, jend)
            jm = j0 + int(np.argmax(s[j0:t1]))
            assert w[jm] == 2.0 ** off


def test_invalid_arguments():
    inp = synth.make_inputs(1, 2, 1, 64, 8, BF16, sharp=False, seed=75)
    q = inp.q[:, :, :4]
    with pytest.raises(ValueError):
        oracle.decode(q, inp.k, inp.v, Sk=64, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE,
                      split_keys=40, Bc=32)  # not a multiple of the tile
    with pytest.raises(ValueError):
        oracle.decode(inp.q, inp.k, inp.v, Sk=32, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE,
                      split_keys=0, Bc=32)  # Sq > Sk
    with pytest.raises(ValueError):
        oracle.decode(q, inp.k, inp.v, Sk=65, dtype=BF16, causal=True, scale=0.3, mode=oracle.H15_TILE,
                      split_keys=0, Bc=32)  # Sk beyond the cache
    with pytest.raises(ValueError):
        oracle.decode(q, inp.k, inp.v, Sk=64, dtype=BF16, causal=True, scale=0.3, mode=oracle.ROWMAX_POT,
                      split_keys=0, Bc=32)
