"""GPU parity of decode over a key/value cache (attn_decode) against the
oracle's decode (oracle.decode): Sq query rows against Sk cached keys with
bottom-right causal alignment, the keys cut into parts that each run the
per-tile recurrence and merge exactly.

Bars as for the forward kernel (parity_helpers): O within 2e-2 max|V| (BF16)
or 6e-2 max|V| (FP8); LSE 1e-3 for the exact control, and for the lattice
weights the median row within 1e-4 and every row within 5e-2 against the
oracle on its own logits; with the oracle fed the GPU's own logits, every W
and P bit for bit and LSE to 1e-5 plus the fp32 summation bound."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth
from parity_helpers import (ALL_MODES, APPROX, BF16, EXACT, FP8, H15, LOGIT_REL, ORACLE_MODE, ORDER, SQ4, SQ8, TOL,
                            assert_close, decoded, dev_tensors, say, scale_of, vmax)

pytestmark = pytest.mark.gpu

BC = 128


def run(inp, Sk, causal, sc, mode, split, out=None, lse=None):
    q, k, v = dev_tensors(inp)
    o, l = pkg.attn_decode(q, k, v, Sk=Sk, causal=causal, scale=sc, exp_mode=mode, split_keys=split,
                           descale=inp.descale, out=out, lse=lse)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), l.cpu().numpy().astype(np.float64)


def ref(inp, Sk, causal, sc, mode, split, rows=None):
    return oracle.decode(inp.q, inp.k, inp.v, Sk=Sk, dtype=inp.dtype, causal=causal, scale=sc,
                         mode=ORACLE_MODE[mode], split_keys=split, descale=inp.descale, Bc=BC, rows=rows)


def check(inp, Sk, causal, sc, mode, split, what):
    o, lse = run(inp, Sk, causal, sc, mode, split)
    o_ref, lse_ref = ref(inp, Sk, causal, sc, mode, split)
    assert_close(inp, o, lse, o_ref, lse_ref, what, mode, flat_lse=True)
    return o, lse


def check_probe(inp, Sk, causal, sc, mode, split, rows):
    """Bit-exact W and P of decode rows (b, h, i) against the oracle fed the
    GPU's logits; the probe's O and LSE equal attn_decode's."""
    q, k, v = dev_tensors(inp)
    dt = inp.dtype
    Sq = inp.q.shape[2]
    G = inp.q.shape[1] // inp.k.shape[1]
    c1 = oracle.c1(sc, inp.descale[0], inp.descale[1])
    o_m, l_m = pkg.attn_decode(q, k, v, Sk=Sk, causal=causal, scale=sc, exp_mode=mode, split_keys=split,
                               descale=inp.descale)
    for (b, h, i) in rows:
        say(f"decode probe dtype={dt} causal={causal} mode={mode} split={split} row ({b},{h},{i})")
        o_p, l_p, s, w, pbits = pkg.attn_decode_probe(q, k, v, Sk=Sk, causal=causal, scale=sc, exp_mode=mode,
                                                      split_keys=split, b=b, h=h, i=i, descale=inp.descale)
        torch.cuda.synchronize()
        assert torch.equal(o_p.view(torch.int16), o_m.view(torch.int16)) and torch.equal(l_p, l_m)
        s, w, pbits = s.cpu().numpy(), w.cpu().numpy(), pbits.cpu().numpy().astype(np.uint32)
        jend = Sk - Sq + i + 1 if causal else Sk
        s_ref = oracle.decode_logits_row(inp.q, inp.k, dt, Sk, b, h, i)
        mag = np.abs(decoded(inp.k[b, h // G, :jend], dt)) @ np.abs(decoded(inp.q[b, h, i], dt))
        assert np.all(np.isneginf(s[jend:]))
        assert np.max(np.abs(s[:jend] - s_ref[:jend]) / np.maximum(mag, 1e-30)) <= LOGIT_REL[dt]
        if mode in APPROX:
            w_ref, p_ref, lse_ref = oracle.decode_row_from_logits(s, jend, c1, dt, BC, split, k=ORDER[mode])
            nparts = 1 if split == 0 or split >= Sk else -(-Sk // split)
            sum_bound = (jend / BC + 64 + 2 * nparts) * 2.0 ** -24
            tol = max(1e-5, 4.0 * float(np.spacing(np.float32(abs(lse_ref))))) + sum_bound
            assert abs(float(l_p[b, h, i]) - lse_ref) <= tol
            assert np.array_equal(w.view(np.uint32), w_ref.view(np.uint32))
            assert np.array_equal(pbits, p_ref)
        else:
            w_ref, _, _ = oracle.decode_row_from_logits(s, jend, c1, dt, BC, split, exact_exp=True)
            assert np.max(np.abs(w - w_ref) / np.maximum(w_ref, 1e-30)) < 4e-7
            wb = w.view(np.uint32).astype(np.uint64)
            enc = (((wb + 0x7FFF + ((wb >> 16) & 1)) >> 16).astype(np.uint32) if dt == BF16
                   else np.array([oracle.e4m3_encode(float(x)) for x in w], np.uint32))
            assert np.array_equal(pbits, enc)


DTD = [(BF16, 128), (FP8, 128), (BF16, 64), (FP8, 64)]


@pytest.mark.parametrize("mode", ALL_MODES)
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("dt,d", DTD)
def test_decode_small_full_parity(dt, d, causal, mode):
    # B2 Hq8 Hkv2, Sq = 3 rows against Sk = 1000 of a 1030-row cache, parts of 256 keys
    inp = synth.make_decode_inputs(2, 8, 2, 3, 1030, d, dt, sharp=True, seed=1100 + d + dt)
    say(f"decode dtype={dt} d={d} causal={causal} mode={mode}")
    check(inp, 1000, causal, scale_of(d), mode, 256, "decode")


@pytest.mark.parametrize("split", [0, 128, 512, 1024])
@pytest.mark.parametrize("Sq", [1, 5])
@pytest.mark.parametrize("mode", [EXACT, H15])
def test_decode_cuts(split, Sq, mode):
    inp = synth.make_decode_inputs(1, 8, 2, Sq, 1000, 128, BF16, sharp=True, seed=1200 + Sq)
    say(f"decode cut split={split} Sq={Sq} mode={mode}")
    check(inp, 1000, True, scale_of(128), mode, split, f"split {split}")


@pytest.mark.parametrize("dt", [BF16, FP8])
@pytest.mark.parametrize("mode", ALL_MODES)
@pytest.mark.parametrize("causal", [False, True])
def test_decode_probe_bit_exact(dt, mode, causal):
    Sq, Sk = 4, 777
    inp = synth.make_decode_inputs(1, 8, 2, Sq, Sk, 128, dt, sharp=True, seed=1300 + dt)
    check_probe(inp, Sk, causal, scale_of(128), mode, 256, ((0, 0, 0), (0, 5, 3), (0, 7, 1)))


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Sk,cap,d", [(1, 1, 1, 1, 1, 1, 128), (1, 2, 1, 1, 129, 200, 64),
                                                  (2, 32, 2, 3, 300, 300, 128), (1, 4, 4, 7, 7, 64, 128),
                                                  (3, 4, 1, 2, 2000, 2048, 64)])
@pytest.mark.parametrize("dt", [BF16, FP8])
def test_decode_edge_shapes(B, Hq, Hkv, Sq, Sk, cap, d, dt):
    # one key; a ragged last tile; several 32-row blocks (G Sq = 48); Sq = Sk;
    # parts whose last one is ragged
    inp = synth.make_decode_inputs(B, Hq, Hkv, Sq, cap, d, dt, sharp=False, seed=1400 + Sk)
    sc = scale_of(d)
    for causal in (False, True):
        for mode in (EXACT, H15, SQ8):
            for split in (0, 128):
                say(f"decode edge B={B} Hq={Hq} Hkv={Hkv} Sq={Sq} Sk={Sk} cap={cap} d={d} dtype={dt} "
                    f"causal={causal} mode={mode} split={split}")
                check(inp, Sk, causal, sc, mode, split, "edge")


@pytest.mark.parametrize("dt", [BF16, FP8])
def test_square_decode_matches_the_forward_kernel(dt):
    # Sq = Sk, one part: the forward kernel's causal rows; the logits come
    # from the same MFMA sequence, so the probe weights agree bit for bit
    S, d = 300, 128
    inp = synth.make_inputs(1, 4, 2, S, d, dt, sharp=True, seed=1500)
    q, k, v = dev_tensors(inp)
    sc = scale_of(d)
    for mode in (EXACT, H15):
        o_d, l_d = pkg.attn_decode(q, k, v, causal=True, scale=sc, exp_mode=mode, split_keys=0, descale=inp.descale)
        o_f, l_f = pkg.attn_fwd_ex(q, k, v, causal=True, scale=sc, exp_mode=mode, descale=inp.descale)
        torch.cuda.synchronize()
        assert float((o_d.float() - o_f.float()).abs().max()) <= TOL[dt] * vmax(inp) / 4
        assert float((l_d - l_f).abs().max()) <= 1e-4
        for (h, i) in ((0, 0), (3, 170), (1, S - 1)):
            _, _, s1, w1, p1 = pkg.attn_decode_probe(q, k, v, causal=True, scale=sc, exp_mode=mode, split_keys=0,
                                                     b=0, h=h, i=i, descale=inp.descale)
            _, _, s2, w2, p2 = pkg.attn_fwd_probe(q, k, v, causal=True, scale=sc, exp_mode=mode, b=0, h=h, row0=i,
                                                  nrows=1, descale=inp.descale)
            torch.cuda.synchronize()
            assert torch.equal(s1, s2[0]) and torch.equal(w1, w2[0]) and torch.equal(p1, p2[0])


def test_cache_rows_beyond_sk_are_never_read():
    Sk, cap = 500, 640
    inp = synth.make_decode_inputs(1, 8, 2, 2, cap, 128, BF16, sharp=True, seed=1600)
    sc = scale_of(128)
    a = run(inp, Sk, True, sc, H15, 256)
    k2, v2 = np.array(inp.k), np.array(inp.v)
    k2[:, :, Sk:] = 0x7FC0  # NaN
    v2[:, :, Sk:] = 0x7FC0
    b = run(synth.Inputs(inp.q, k2, v2, inp.descale, BF16), Sk, True, sc, H15, 256)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_deterministic_and_every_row_written():
    inp = synth.make_decode_inputs(4, 32, 8, 2, 3000, 128, FP8, sharp=True, seed=1700)
    q, k, v = dev_tensors(inp)
    sc = scale_of(128)
    for split in (0, 384):
        o1 = torch.full((4, 32, 2, 128), float("nan"), dtype=torch.bfloat16, device="cuda:0")
        l1 = torch.full((4, 32, 2), float("nan"), dtype=torch.float32, device="cuda:0")
        pkg.attn_decode(q, k, v, causal=True, scale=sc, exp_mode=H15, split_keys=split, descale=inp.descale,
                        out=o1, lse=l1)
        o2, l2 = pkg.attn_decode(q, k, v, causal=True, scale=sc, exp_mode=H15, split_keys=split,
                                 descale=inp.descale)
        torch.cuda.synchronize()
        assert not torch.isnan(o1.float()).any() and not torch.isnan(l1).any()
        assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)


@pytest.mark.parametrize("dt,d", [(BF16, 64), (FP8, 128)])
def test_writes_stay_inside_outputs(dt, d):
    # O, LSE and the workspace as views into larger NaN-filled buffers: the
    # guard regions on both sides stay untouched, with one part and with
    # several (the parts' partial results, then the merge)
    B, Hq, Hkv, Sq, Sk = 2, 8, 2, 3, 1000
    inp = synth.make_decode_inputs(B, Hq, Hkv, Sq, Sk, d, dt, sharp=True, seed=1750 + d)
    q, k, v = dev_tensors(inp)
    sc = scale_of(d)
    G = 4096
    n_o, n_l = B * Hq * Sq * d, B * Hq * Sq
    for split in (0, 256):
        say(f"decode guard dtype={dt} d={d} split={split}")
        ob = torch.full((G + n_o + G,), float("nan"), dtype=torch.bfloat16, device="cuda:0")
        lb = torch.full((G + n_l + G,), float("nan"), dtype=torch.float32, device="cuda:0")
        need = pkg.attn_decode_workspace_bytes(B, Hq, Sq, Sk, d, split)
        wb = torch.full((G + max(need, 16) + G,), 0x5A, dtype=torch.uint8, device="cuda:0")
        o, lse = ob[G:G + n_o].view(B, Hq, Sq, d), lb[G:G + n_l].view(B, Hq, Sq)
        pkg.attn_decode(q, k, v, causal=True, scale=sc, exp_mode=H15, split_keys=split, descale=inp.descale,
                        out=o, lse=lse, workspace=wb[G:G + max(need, 16)])
        o2, l2 = pkg.attn_decode(q, k, v, causal=True, scale=sc, exp_mode=H15, split_keys=split,
                                 descale=inp.descale)
        torch.cuda.synchronize()
        assert torch.isnan(ob[:G].float()).all() and torch.isnan(ob[G + n_o:].float()).all()
        assert torch.isnan(lb[:G]).all() and torch.isnan(lb[G + n_l:]).all()
        assert (wb[:G] == 0x5A).all() and (wb[G + max(need, 16):] == 0x5A).all()
        assert torch.equal(o.view(torch.int16), o2.view(torch.int16)) and torch.equal(lse, l2)


DECODE_FULL = [("bf16", BF16), ("fp8", FP8)]


@pytest.mark.parametrize("name,dt", DECODE_FULL)
@pytest.mark.parametrize("mode", [EXACT, H15])
def test_decode_full_size(name, dt, mode):
    # the decode benchmark's shape: B16 Hq32 Hkv8, one query row per head
    # against an 8K cache, the library's proposed cut
    B, Hq, Hkv, Sq, Sk, d = 16, 32, 8, 1, 8192, 128
    say(f"decode full-size {name} mode={mode}: inputs")
    inp = synth.make_decode_inputs(B, Hq, Hkv, Sq, Sk, d, dt, sharp=True, seed=1800 + dt)
    sc = scale_of(d)
    split = pkg.attn_decode_split_keys(B, Hq, Hkv, Sq, Sk, d, dt)
    assert split > 0 and split % BC == 0
    o, lse = run(inp, Sk, True, sc, mode, split)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    assert np.max(np.abs(o)) <= vmax(inp) * (1 + 2 ** -7)
    rows = np.unique(np.concatenate([np.arange(0, B * Hq, 7), [B * Hq - 1]]))
    say(f"decode full-size {name} mode={mode}: oracle on {len(rows)} rows")
    o_ref, lse_ref = ref(inp, Sk, True, sc, mode, split, rows=rows)
    assert_close(inp, o.reshape(-1, d)[rows], lse.reshape(-1)[rows], o_ref, lse_ref, "decode full", mode,
                 flat_lse=True)
    check_probe(inp, Sk, True, sc, mode, split, ((B - 1, Hq - 1, 0), (3, 9, 0)))
