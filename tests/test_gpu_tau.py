"""GPU parity of the conditional rescale (App. B.2, "Conditional rescaling
moves the anchor"): with tau = 8 (the BF16 FlashAttention-4 setting) the
running max moves only when a row's maximum grows by more than 8 octaves,
decided per row or shared by the wave's 32 rows (rescale_per_wave).  Same
bars as the other modes: O within 2e-2 max|V| and LSE as for H15 against the
oracle on its own logits; W, P and LSE bit-identical (LSE to 1e-5) against
the oracle fed the GPU's own logits and, per wave, the group decision taken
from those logits."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth
from parity_helpers import (ALL_MODES, APPROX, EXACT, H15, ORACLE_MODE, ORDER, SQ4, assert_close, dev_tensors,
                            say, scale_of)

pytestmark = pytest.mark.gpu

BF16 = synth.BF16
TAU = 8.0


def rising_inputs(S, d, Hq=4, Hkv=2, seed=700):
    """Keys whose norm grows with their index, so a row's running maximum
    keeps rising across tiles: under tau = 8 some tiles move the anchor and
    some keep it."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((1, Hq, S, d)).astype(np.float32)
    k = rng.standard_normal((1, Hkv, S, d)).astype(np.float32)
    k *= (0.3 + 2.5 * np.arange(S, dtype=np.float32) / S)[None, None, :, None]
    v = rng.standard_normal((1, Hkv, S, d)).astype(np.float32)
    return synth.Inputs(synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v), (1.0, 1.0, 1.0), BF16)


def run(inp, causal, sc, mode, tau, per_wave):
    q, k, v = dev_tensors(inp)
    o, lse = pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, tau=tau, tau_per_wave=per_wave)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("per_wave", [False, True])
@pytest.mark.parametrize("mode", ALL_MODES)
@pytest.mark.parametrize("d,causal,S", [(128, True, 700), (128, False, 300), (64, True, 300)])
def test_tau_full_parity(d, causal, S, mode, per_wave):
    inp = rising_inputs(S, d)
    sc = scale_of(d)
    say(f"tau={TAU} per_wave={per_wave} d={d} causal={causal} S={S} mode={mode}")
    o, lse = run(inp, causal, sc, mode, TAU, per_wave)
    o_ref, lse_ref = oracle.attn(inp.q, inp.k, inp.v, dtype=BF16, causal=causal, scale=sc, mode=ORACLE_MODE[mode],
                                 Bc=pkg.attn_tile_bc(), tau=TAU, tau_group=32 if per_wave else 1)
    assert_close(inp, o, lse, o_ref, lse_ref, "tau", mode, flat_lse=True)
    if mode in APPROX:
        # the threshold changes the approximate result somewhere
        o0, _ = run(inp, causal, sc, mode, 0.0, False)
        assert np.any(o0 != o)


@pytest.mark.parametrize("per_wave", [False, True])
@pytest.mark.parametrize("mode", [H15, SQ4])
@pytest.mark.parametrize("causal", [False, True])
def test_tau_probe_bit_exact(causal, mode, per_wave):
    S, d = 600, 128
    inp = rising_inputs(S, d, Hq=2, Hkv=1, seed=701)
    sc = scale_of(d)
    q, k, v = dev_tensors(inp)
    c1 = oracle.c1(sc)
    Bc = pkg.attn_tile_bc()
    moved = kept = 0
    for (h, r0) in ((0, 0), (1, 256), (0, 544)):  # rows [r0, r0 + 32): one wave's rows
        n = min(32, S - r0)
        say(f"tau probe causal={causal} mode={mode} per_wave={per_wave} head {h} rows {r0}+{n}")
        _, lse_p, s, w, pbits = pkg.attn_fwd_probe(q, k, v, causal=causal, scale=sc, exp_mode=mode, b=0, h=h,
                                                   row0=r0, nrows=n, tau=TAU, tau_per_wave=per_wave)
        torch.cuda.synchronize()
        s, w, pbits, lse_p = s.cpu().numpy(), w.cpu().numpy(), pbits.cpu().numpy().astype(np.uint32), lse_p.cpu().numpy()
        sv = np.where(np.isneginf(s), np.float32(0.0), s)  # masked logits are never read
        move = oracle.group_moves_from_logits(sv, r0, causal, c1, Bc, TAU) if per_wave else None
        if move is not None:
            nt = (r0 + n - 1) // Bc + 1 if causal else (S + Bc - 1) // Bc
            moved += int(move[1:nt].sum())
            kept += int((move[1:nt] == 0).sum())
        for r in range(n):
            i = r0 + r
            if per_wave:
                w_ref, p_ref, lse_ref = oracle.sq_row_from_logits_moves(sv[r], i, causal, c1, BF16, Bc, ORDER[mode],
                                                                        move)
            else:
                w_ref, p_ref, lse_ref = oracle.sq_row_from_logits(sv[r], i, causal, c1, BF16, Bc, k=ORDER[mode],
                                                                  tau=TAU)
            assert np.array_equal(w[r].view(np.uint32), w_ref.view(np.uint32)), f"row {i}"
            assert np.array_equal(pbits[r], p_ref), f"row {i}"
            assert abs(lse_p[0, h, i] - lse_ref) <= 1e-5, f"row {i}"
    if per_wave and not causal:
        # both outcomes of the shared decision occur in these rows
        assert moved > 0 and kept > 0


def test_tau_zero_is_the_default():
    inp = rising_inputs(300, 128)
    sc = scale_of(128)
    for mode in (H15, EXACT):
        a = run(inp, True, sc, mode, 0.0, True)
        q, k, v = dev_tensors(inp)
        o, lse = pkg.attn_fwd(q, k, v, causal=True, scale=sc, exp_mode=mode)
        torch.cuda.synchronize()
        assert np.array_equal(a[0], o.float().cpu().numpy().astype(np.float64))
        assert np.array_equal(a[1], lse.cpu().numpy().astype(np.float64))
