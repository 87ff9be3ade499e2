"""Pins of the oracle's Rowmax-H15 weight function and operand codecs.

The oracle is checked against what the paper fixes (its worked example, its
constants, the closed form H = S o Q_1/2 and the octave-error envelope of
App. B.1) and against library routines (torch's bfloat16 / float8_e4m3fn
casts), never against itself."""
import json
import math
from pathlib import Path

import numpy as np
import pytest
import torch

import oracle

FACTS = json.loads((Path(__file__).parent / "golden" / "h15_paper_facts.json").read_text())


def f32_bits(x: float) -> int:
    return int(np.array([x], np.float32).view(np.uint32)[0])


def test_worked_example_from_paper():
    ex = FACTS["worked_example"]
    # y is the doubled input 2x; an integer y is already RNE-rounded: n = y.
    assert oracle.h15_weight(float(ex["n"])) == ex["weight"]
    assert oracle.h15_ideal(float(ex["n"])) == ex["weight"]


def test_constants_from_paper():
    c = FACTS["implementation_constants"]
    assert f32_bits(c["magic_add_value"]) == int(c["magic_add_bits"], 16)
    assert c["magic_add_value"] == 2.0 ** 23 + 2.0 ** 22
    assert f32_bits(1.0) == int(c["one_bits"], 16)
    # Clamp at -252: every input below gives the weight of -252, 2^-126.
    for y in (-252.0, -252.4, -253.0, -1000.0, -1e30, -float(np.finfo(np.float32).max)):
        assert oracle.h15_weight(y) == 2.0 ** -126


@pytest.mark.parametrize("n", range(-252, 256))
def test_even_odd_lattice_closed_form(n):
    # Eq. (h15): even n -> 2^(n/2), odd n -> 1.5 * 2^floor(n/2).
    k = n // 2  # floor toward -inf
    want = 2.0 ** k if n % 2 == 0 else 1.5 * 2.0 ** k
    assert oracle.h15_weight(float(n)) == want


def test_exhaustive_bit_form_equals_closed_form():
    # App. B.1: the add/shift form equals S(Q_1/2(x)); checked on every fp32 y
    # in [-300, 255] (beyond the paper's 2,295,040 sampled inputs).
    bad, n = oracle.h15_exhaustive(-300.0, 255.0)
    assert n > 2_200_000_000
    assert bad == 0


def test_schraudolph_identity_on_half_integers():
    # S(x) = 2^floor(x) (1 + x - floor(x)), H(x) = S(Q_1/2(x)), Q_1/2(x) = RNE(2x)/2.
    rng = np.random.default_rng(0)
    ys = np.concatenate([rng.uniform(-250, 30, 20000), np.arange(-250, 30, 0.5)]).astype(np.float32)
    for y in ys[:5000]:
        q = np.rint(np.float64(y)) / 2.0  # numpy rint: round half to even
        s = 2.0 ** math.floor(q) * (1.0 + q - math.floor(q))
        assert oracle.h15_weight(float(y)) == s


def test_octave_error_envelope():
    env = FACTS["octave_error_envelope"]
    lo, hi = env["lower"], math.log2(1.5) - 0.25
    assert abs(hi - env["upper_printed"]) < 5e-6
    rng = np.random.default_rng(1)
    ys = rng.uniform(-250.0, 20.0, 200000).astype(np.float32)
    ys = np.concatenate([ys, np.arange(-250.0, 20.0, 0.25, dtype=np.float32)])
    errs = np.array([math.log2(oracle.h15_weight(float(y))) - float(y) / 2.0 for y in ys])
    assert errs.min() >= lo - 1e-12
    assert errs.max() <= hi + 1e-12
    # both ends are (nearly) reached
    assert errs.min() < lo + 1e-3 and errs.max() > hi - 1e-3


def test_every_weight_on_the_lattice():
    rng = np.random.default_rng(2)
    ys = rng.uniform(-300.0, 40.0, 100000).astype(np.float32)
    for y in ys[:20000]:
        b = f32_bits(oracle.h15_weight(float(y)))
        assert b & 0x3FFFFF == 0  # mantissa holds at most its top bit: {1, 1.5} x 2^k


def test_output_log_spacing():
    sp = FACTS["output_log_spacing"]["spacings"]
    w = [oracle.h15_weight(float(n)) for n in range(-20, 1)]
    gaps = np.diff(np.log2(w))
    for i, g in enumerate(gaps):
        want = math.log2(1.5) if i % 2 == 0 else 1 - math.log2(1.5)
        assert abs(g - want) < 1e-12
    assert abs(math.log2(1.5) - sp[0]) < 1e-3 and abs(1 - math.log2(1.5) - sp[1]) < 1e-3


def test_rne_ties_go_to_even():
    # y = k + 1/2 rounds to the even neighbour (App. B.1: RNE).
    assert oracle.h15_weight(-2.5) == oracle.h15_weight(-2.0)
    assert oracle.h15_weight(-3.5) == oracle.h15_weight(-4.0)
    assert oracle.h15_weight(0.5) == 1.0
    assert oracle.h15_weight(1.5) == 2.0


def test_bf16_decode_vs_torch():
    bits = np.arange(0, 1 << 16, 7, dtype=np.int64)
    t = torch.tensor(bits.astype(np.int16), dtype=torch.int16).view(torch.bfloat16).double().numpy()
    for b, want in zip(bits[::50], t[::50]):
        got = oracle.bf16_value(int(b))
        assert (got == want) or (math.isnan(got) and math.isnan(want))


def test_e4m3_decode_vs_torch():
    codes = np.arange(256, dtype=np.uint8)
    t = torch.tensor(codes).view(torch.float8_e4m3fn).double().numpy()
    for c in codes:
        got = oracle.e4m3_value(int(c))
        assert (got == t[c]) or (math.isnan(got) and math.isnan(t[c]))
    assert oracle.e4m3_value(0x7E) == 448.0
    assert oracle.e4m3_value(0x01) == 2.0 ** -9


def test_e4m3_encode_vs_torch():
    rng = np.random.default_rng(3)
    xs = np.concatenate([
        rng.uniform(-448, 448, 20000),
        2.0 ** rng.uniform(-12, 8.8, 20000),
        np.arange(0, 64) * 2.0 ** -10,  # exact ties in the subnormal range
        [0.0, 448.0, 2.0 ** -6, 2.0 ** -9, 1.5 * 2.0 ** -9],
    ]).astype(np.float32)
    want = torch.tensor(xs).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = np.array([oracle.e4m3_encode(float(x)) for x in xs], np.uint8)
    assert np.array_equal(got, want)
    # saturation above the largest finite value
    assert oracle.e4m3_encode(1e6) == 0x7E and oracle.e4m3_encode(-1e6) == 0xFE


def test_h15_lattice_is_exact_in_storage_types():
    # Lattice weights are normal fp32 values with a 2-bit significand, so
    # bf16 holds them exactly, and e4m3 holds every one from 2^-6 to 2^8.
    for n in range(-252, 17):
        w = oracle.h15_weight(float(n))
        b = f32_bits(w)
        assert b & 0xFFFF == 0  # bf16 exact
        if -12 <= n <= 16:
            assert oracle.e4m3_value(oracle.e4m3_encode(w)) == w


def test_c1_doubling_is_exact():
    for d in (64, 128):
        c1 = oracle.c1(1.0 / math.sqrt(d))
        assert np.float32(2.0) * np.float32(c1) == np.float32(2.0 * c1)
    assert oracle.c1(1.0 / math.log2(math.e)) == 1.0
