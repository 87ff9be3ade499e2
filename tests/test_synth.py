"""The seeded input generator: determinism, sharp-key recipe and the operand
codecs against torch's casts."""
import numpy as np
import torch

from paper_2609_33586_amd import synth


def test_bf16_bits_match_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 100
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(synth.bf16_bits(x), want)
    assert np.array_equal(synth.bf16_decode(want), torch.from_numpy(want.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_e4m3_codes_match_torch():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.uniform(-448, 448, 50000), 2.0 ** rng.uniform(-12, 8.8, 50000)]).astype(np.float32)
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(synth.e4m3_codes(x), want)
    codes = np.arange(256, dtype=np.uint8)
    dec = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    fin = ~np.isnan(dec)
    assert np.array_equal(synth.e4m3_decode(codes)[fin], dec[fin])


def test_deterministic_and_sharp_recipe():
    a = synth.make_inputs(1, 2, 1, 200, 8, synth.BF16, sharp=True, seed=5)
    b = synth.make_inputs(1, 2, 1, 200, 8, synth.BF16, sharp=True, seed=5)
    assert all(np.array_equal(x, y) for x, y in ((a.q, b.q), (a.k, b.k), (a.v, b.v)))
    # redo the recipe by hand: 2% of key rows scaled by 4
    rng = np.random.Generator(np.random.PCG64(5))
    q = rng.standard_normal((1, 2, 200, 8), dtype=np.float32)
    k = rng.standard_normal((1, 1, 200, 8), dtype=np.float32)
    rng.standard_normal((1, 1, 200, 8), dtype=np.float32)
    idx = rng.permutation(200)[:4]
    k[0, 0, idx] *= 4
    assert np.array_equal(a.k, synth.bf16_bits(k)) and np.array_equal(a.q, synth.bf16_bits(q))


def test_fp8_per_tensor_scale():
    inp = synth.make_inputs(1, 1, 1, 64, 16, synth.FP8_E4M3, sharp=False, seed=6)
    for codes, s in zip((inp.q, inp.k, inp.v), inp.descale):
        assert codes.dtype == np.uint8 and s > 0
        assert np.max(np.abs(synth.e4m3_decode(codes))) == 448.0  # amax maps to the largest code


def test_workload_table():
    w = synth.WORKLOADS["causal_fp8_b2_h32kv8_s8192_d128_sharp"]
    assert (w.B, w.Hq, w.Hkv, w.S, w.d, w.causal, w.dtype) == (2, 32, 8, 8192, 128, True, synth.FP8_E4M3)
    assert abs(w.flops() - 2 * 2 * 32 * 8192 ** 2 * 128) < 1
