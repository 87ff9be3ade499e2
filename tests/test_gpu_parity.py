"""GPU parity: the HIP kernels (through the C ABI) against the CPU oracle.

Bars (parity_helpers): max |O_gpu - O_oracle| <= 2e-2 max|V| for BF16
operands and 6e-2 max|V| for FP8, with V the dequantised values.  EXACT mode
is compared with the oracle's exact softmax on its own (fp64) logits, the
lattice weights (H15, S(Q_{1/4}), S(Q_{1/8})) with the oracle's per-tile
recurrence on its own fp32 logits.  LSE: 1e-3 for EXACT; for the lattice
weights each row within the bound that the GPU's logit accuracy implies
(lse_bound_lattice) and the median row within 1e-4; against the oracle fed
the GPU's own logits to 1e-5 plus the fp32 summation bound of l, with the
weights and stored P bit for bit.  Rowmax-PoT (BF16) is held to the fp64
operator of Eq. (rowmax-pot) (LSE: median 1e-4, every row 5e-2), with its W
and P bit-exact against the row form of the oracle fed the GPU's logits."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth
from parity_helpers import (ALL_MODES, APPROX, BF16, EXACT, FP8, H15, ORDER, POT, SQ4, SQ8, TOL, assert_close,
                            check_probe, dev_tensors, gpu_run, oracle_run, say, scale_of, stratified_rows, vmax)

pytestmark = pytest.mark.gpu

SMALL = [(dt, d, causal, S) for dt in (BF16, FP8) for d in (64, 128) for causal in (False, True)
         for S in (256, 300)]


@pytest.mark.parametrize("mode", ALL_MODES)
@pytest.mark.parametrize("dt,d,causal,S", SMALL)
def test_small_full_parity(dt, d, causal, S, mode):
    inp = synth.make_inputs(1, 4, 2, S, d, dt, sharp=True, seed=100 + S + d)
    sc = scale_of(d)
    say(f"small dtype={dt} d={d} causal={causal} S={S} mode={mode}")
    o, lse = gpu_run(inp, causal, sc, mode)
    o_ref, lse_ref = oracle_run(inp, causal, sc, mode)
    assert_close(inp, o, lse, o_ref, lse_ref, "full", mode, causal=causal, sc=sc)


@pytest.mark.parametrize("dt", [BF16, FP8])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("mode", ALL_MODES)
def test_probe_weights_bit_exact(dt, causal, mode):
    S, d = 520, 128
    inp = synth.make_inputs(1, 4, 1, S, d, dt, sharp=True, seed=201)
    check_probe(inp, S, d, dt, causal, mode, scale_of(d), ((0, 0, 0, 40), (0, 3, 250, 40), (0, 2, S - 37, 37)))


@pytest.mark.parametrize("S", [576, 610])
@pytest.mark.parametrize("dt", [BF16, FP8])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("mode", ALL_MODES)
def test_probe_ragged_tail_across_key_halves(S, dt, causal, mode):
    # The last key tile ends exactly at its 64-key half (S = 576) or inside
    # the second half (S = 610, 98 keys): at fp8 the kernel finishes the two
    # halves of a tile's weights at different points of the PV product.
    d = 128
    inp = synth.make_inputs(1, 4, 2, S, d, dt, sharp=True, seed=700 + S)
    check_probe(inp, S, d, dt, causal, mode, scale_of(d), ((0, 1, S - 70, 70), (0, 2, 100, 30)))


@pytest.mark.parametrize("mode", ALL_MODES)
@pytest.mark.parametrize("dt,d", [(BF16, 64), (BF16, 128), (FP8, 64), (FP8, 128)])
@pytest.mark.parametrize("causal", [False, True])
def test_equal_logits_closed_form(mode, dt, d, causal):
    # K = 0 makes every logit 0: each visible key gets the same weight (2^off
    # in every mode, exact at the anchor), so O is the plain mean of the
    # visible V rows and LSE = ln(number of visible keys).  No oracle needed.
    S = 300
    inp = synth.make_inputs(1, 4, 2, S, d, dt, sharp=False, seed=900 + d)
    inp.k[...] = 0
    o, lse = gpu_run(inp, causal, scale_of(d), mode)
    vdec = synth.bf16_decode(inp.v) if dt == BF16 else synth.e4m3_decode(inp.v) * inp.descale[2]
    vdec = vdec.astype(np.float64)
    G = 2
    cnt = np.arange(1, S + 1, dtype=np.float64) if causal else np.full(S, float(S))
    for h in range(4):
        vh = vdec[0, h // G]
        mean = np.cumsum(vh, axis=0) / cnt[:, None] if causal else np.broadcast_to(vh.mean(axis=0), vh.shape)
        assert np.max(np.abs(o[0, h] - mean)) <= TOL[dt] * vmax(inp), f"head {h}"
        dl = np.abs(lse[0, h] - np.log(cnt)) - 4.0 * np.spacing(np.log(cnt).astype(np.float32))
        assert np.max(dl) <= 1e-5, f"head {h}"


@pytest.mark.parametrize("mode", ALL_MODES)
@pytest.mark.parametrize("dt,d", [(BF16, 64), (BF16, 128), (FP8, 64), (FP8, 128)])
@pytest.mark.parametrize("causal", [False, True])
def test_dominant_key_closed_form(mode, dt, d, causal):
    # K = 12 Q (MHA): each row's own key outscores every other by at least 40
    # octaves (83 at d = 128), so every other weight is below 2^-40 of it; O is
    # the row's own V row and LSE its own scaled logit.  No oracle needed.
    S = 300
    base = synth.make_inputs(1, 2, 2, S, d, dt, sharp=False, seed=950 + d)
    qdec = (synth.bf16_decode(base.q) if dt == BF16 else synth.e4m3_decode(base.q) * base.descale[0])
    kf = (12.0 * qdec).astype(np.float32)
    if dt == BF16:
        inp = synth.Inputs(base.q, synth.bf16_bits(kf), base.v, (1.0, 1.0, 1.0), BF16)
    else:
        kc, ks = synth.quantize_e4m3(kf)
        inp = synth.Inputs(base.q, kc, base.v, (base.descale[0], ks, base.descale[2]), dt)
    o, lse = gpu_run(inp, causal, scale_of(d), mode)
    qd = qdec.astype(np.float64)
    kd = (synth.bf16_decode(inp.k) if dt == BF16 else synth.e4m3_decode(inp.k) * inp.descale[1]).astype(np.float64)
    vd = (synth.bf16_decode(inp.v) if dt == BF16 else synth.e4m3_decode(inp.v) * inp.descale[2]).astype(np.float64)
    sc = scale_of(d)
    for h in range(2):
        logits = qd[0, h] @ kd[0, h].T
        if causal:
            logits = np.where(np.tril(np.ones((S, S), bool)), logits, -np.inf)
        assert np.all(np.argmax(logits, axis=1) == np.arange(S))
        assert np.max(np.abs(o[0, h] - vd[0, h])) <= TOL[dt] * vmax(inp), f"head {h}"
        lse_ref = sc * np.diagonal(logits)
        # the logit's own accuracy: fp32 sums at BF16; the FP8 matrix core's
        # accumulation agrees to about 2^-13 of sum |q k|, which here (all
        # products positive) is 2^-13 of the logit itself
        rel = 2.0 ** -12 if dt == FP8 else 1e-5
        assert np.all(np.abs(lse[0, h] - lse_ref) <= rel * np.abs(lse_ref) + 1e-5), f"head {h}"


@pytest.mark.parametrize("side", ["below", "above"])
@pytest.mark.parametrize("mode", APPROX)
def test_fp8_saturated_logits_at_the_narrow_clamp_limit(side, mode):
    # Every operand at +-448 puts the raw logits at +-d 448^2, the ends of the
    # bound the launcher uses to choose the 16-bit lane clamp (|y| < 2^15).
    # The descales place that bound just below 2^15 (lane clamp, rounded
    # exponents down to about -32000) or just above it (FP32 clamp); both
    # must give the oracle's bits.
    S, d, k = 200, 128, ORDER[mode]
    sc = scale_of(d)
    target = 32000.0 if side == "below" else 33500.0
    c1_unit = oracle.c1(sc)
    delta = math.sqrt((target - 8.0 * 2 ** k) / (2.0 * 2 ** k * c1_unit * d * 448.0 ** 2))
    bound = 2.0 * 2 ** k * oracle.c1(sc, delta, delta) * d * 448.0 ** 2 * (1 + 1e-5) + 8.0 * 2 ** k
    assert (bound < 32767.0) == (side == "below")
    rng = np.random.default_rng(220 + k)
    q = np.full((1, 1, S, d), 448.0, np.float32)
    kk = np.where(rng.random((1, 1, S, d)) < 0.5, 448.0, -448.0).astype(np.float32)
    kk[0, 0, ::7] = 448.0    # aligned keys: the row maximum d 448^2
    kk[0, 0, 3::7] = -448.0  # anti-aligned keys: y near -2 ck d 448^2
    vv = rng.integers(-3, 4, (1, 1, S, d)).astype(np.float32)
    inp = synth.Inputs(synth.e4m3_codes(q), synth.e4m3_codes(kk), synth.e4m3_codes(vv), (delta, delta, 1.0), FP8)
    check_probe(inp, S, d, FP8, True, mode, sc, ((0, 0, 0, 40), (0, 0, S - 40, 40)))
    o, lse = gpu_run(inp, True, sc, mode)
    o_ref, lse_ref = oracle_run(inp, True, sc, mode)
    assert_close(inp, o, lse, o_ref, lse_ref, f"saturated logits, bound {bound:.0f}", mode, causal=True, sc=sc)


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("mode", APPROX)
def test_fp8_unit_descales_float_clamp_path(causal, mode):
    # With unit descales the FP8 exponent bound 2 * 2^k c1 d 448^2 exceeds
    # 2^15, so the library takes the FP32 clamp form instead of the 16-bit
    # lane one: the same bits are required.
    S, d = 300, 128
    rng = np.random.default_rng(210)
    x = [rng.integers(-3, 4, shape).astype(np.float32) for shape in ((1, 2, S, d), (1, 1, S, d), (1, 1, S, d))]
    inp = synth.Inputs(*(synth.e4m3_codes(a) for a in x), (1.0, 1.0, 1.0), FP8)
    sc = scale_of(d)
    assert 2.0 * 2.0 ** ORDER[mode] * oracle.c1(sc) * d * 448.0 ** 2 > 2.0 ** 15
    check_probe(inp, S, d, FP8, causal, mode, sc, ((0, 0, 0, 30), (0, 1, S - 30, 30)))
    o, lse = gpu_run(inp, causal, sc, mode)
    o_ref, lse_ref = oracle_run(inp, causal, sc, mode)
    assert_close(inp, o, lse, o_ref, lse_ref, "unit descales", mode, causal=causal, sc=sc)


@pytest.mark.parametrize("dt", [BF16, FP8])
@pytest.mark.parametrize("S", [128, 512])
def test_one_hot_value_gates(dt, S):
    # App. B.2 gate design: one-hot V exposes the probabilities; single-tile
    # (S = 128) and multi-tile (S = 512) causal gates, H15 mode.
    d = 128
    rng = np.random.default_rng(300 + S)
    base = synth.make_inputs(1, 2, 2, S, d, dt, sharp=True, seed=301 + S)
    sc = scale_of(d)
    for blk in range(S // d):
        vv = np.zeros((1, 2, S, d), np.float32)
        for c in range(d):
            vv[0, :, blk * d + c, c] = 1.0
        vcodes = synth.bf16_bits(vv) if dt == BF16 else synth.e4m3_codes(vv)
        inp = synth.Inputs(base.q, base.k, vcodes, (base.descale[0], base.descale[1], 1.0), dt)
        say(f"one-hot gate dtype={dt} S={S} block {blk}")
        o, lse = gpu_run(inp, True, sc, H15)
        o_ref, lse_ref = oracle_run(inp, True, sc, H15)
        assert_close(inp, o, lse, o_ref, lse_ref, "one-hot", H15, causal=True, sc=sc)
        # read back probabilities and check the normalized octave bound against
        # exact softmax (App. B.2: +-0.585 plus storage rounding allowances)
        p_gpu = o[0, :, :, :]
        o_ex, _ = oracle_run(inp, True, sc, EXACT)
        p_ex = o_ex[0]
        m = (p_ex > 1e-3) & (p_gpu > 0)
        r = np.log2(p_gpu[m] / p_ex[m])
        allow = 0.585 + (0.01 if dt == BF16 else 0.09)
        assert np.max(np.abs(r)) <= allow


WORKLOADS = list(synth.WORKLOADS.values())


FULL_CASES = [(w, m) for w in WORKLOADS for m in (EXACT, H15)] + [
    (synth.WORKLOADS[n], m) for n in ("causal_fp8_b2_h32kv8_s8192_d128_sharp", "causal_bf16_b4_h32kv8_s2048_d128_sharp")
    for m in (SQ4, SQ8)]


@pytest.mark.parametrize("w,mode", FULL_CASES, ids=[f"{w.name}-{m}" for w, m in FULL_CASES])
def test_full_size_sampled_rows(w, mode):
    say(f"full-size {w.name} mode={mode}: generating inputs")
    inp = synth.workload_inputs(w)
    sc = scale_of(w.d)
    tensors = dev_tensors(inp)
    say(f"full-size {w.name} mode={mode}: GPU run")
    o, lse = gpu_run(inp, w.causal, sc, mode, tensors)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    # O is a convex combination of V rows (times the descale)
    assert np.max(np.abs(o)) <= vmax(inp) * (1 + 2 ** -7)
    rows = stratified_rows(w.B, w.Hq, w.S, 256 if w.dtype == BF16 else 128, seed=7)
    say(f"full-size {w.name} mode={mode}: oracle on {len(rows)} rows")
    o_ref, lse_ref = oracle_run(inp, w.causal, sc, mode, rows=rows)
    assert_close(inp, o.reshape(-1, w.d)[rows], lse.reshape(-1)[rows], o_ref, lse_ref, "sampled rows", mode,
                 causal=w.causal, sc=sc, rows=rows)


@pytest.mark.parametrize("dt,S,causal", [(FP8, 1 << 20, False), (BF16, 1 << 19, True)])
def test_long_sequence_offsets(dt, S, causal):
    # One head whose K/V span 128 MiB: the 32-bit per-head byte offsets of
    # the tile copies reach 2^27 (the launcher accepts up to 2^31), the
    # 64-bit row offsets of Q and O pass 2^27 elements.  Rows from the first,
    # middle and last tiles against the oracle; probe weights bit-exact on
    # the last rows.
    d = 128
    say(f"long sequence dt={dt} S={S} causal={causal}: generating inputs")
    inp = synth.make_inputs(1, 1, 1, S, d, dt, sharp=True, seed=4321)
    sc = scale_of(d)
    tensors = dev_tensors(inp)
    say(f"long sequence dt={dt} S={S}: GPU run")
    o, lse = gpu_run(inp, causal, sc, H15, tensors)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    rows = np.array([0, 127, 128, S // 2 - 1, S // 2, S - 129, S - 128, S - 1])
    say(f"long sequence dt={dt} S={S}: oracle on {len(rows)} rows")
    o_ref, lse_ref = oracle_run(inp, causal, sc, H15, rows=rows)
    assert_close(inp, o.reshape(-1, d)[rows], lse.reshape(-1)[rows], o_ref, lse_ref, "long sequence rows", H15,
                 causal=causal, sc=sc, rows=rows)
    check_probe(inp, S, d, dt, causal, H15, sc, ((0, 0, S - 3, 3),))


@pytest.mark.parametrize("mode", APPROX)
@pytest.mark.parametrize("w", [x for x in WORKLOADS if x.S >= 8192], ids=lambda x: x.name)
def test_full_size_probe_bit_exact(w, mode):
    inp = synth.workload_inputs(w)
    sc = scale_of(w.d)
    q, k, v = dev_tensors(inp)
    c1 = oracle.c1(sc, inp.descale[0], inp.descale[1])
    b, h, r0, n = w.B - 1, w.Hq - 1, w.S - 40, 40
    say(f"full-size probe {w.name} mode={mode} rows {r0}+{n}")
    _, _, s, wt, pbits = pkg.attn_fwd_probe(q, k, v, causal=w.causal, scale=sc, exp_mode=mode, b=b, h=h,
                                            row0=r0, nrows=n, descale=inp.descale)
    torch.cuda.synchronize()
    s, wt, pbits = s.cpu().numpy(), wt.cpu().numpy(), pbits.cpu().numpy().astype(np.uint32)
    for r in range(0, n, 7):
        w_ref, p_ref, _ = oracle.sq_row_from_logits(s[r], r0 + r, w.causal, c1, w.dtype, pkg.attn_tile_bc(),
                                                    k=ORDER[mode])
        assert np.array_equal(wt[r].view(np.uint32), w_ref.view(np.uint32))
        assert np.array_equal(pbits[r], p_ref)


@pytest.mark.parametrize("dt", [BF16, FP8])
def test_deterministic_and_every_row_written(dt):
    inp = synth.make_inputs(2, 8, 2, 700, 128, dt, sharp=True, seed=400)
    sc = scale_of(128)
    q, k, v = dev_tensors(inp)
    for causal in (False, True):
        for mode in (EXACT, H15):
            say(f"determinism dtype={dt} causal={causal} mode={mode}")
            o1 = torch.full((2, 8, 700, 128), float("nan"), dtype=torch.bfloat16, device="cuda:0")
            l1 = torch.full((2, 8, 700), float("nan"), dtype=torch.float32, device="cuda:0")
            pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, descale=inp.descale, out=o1, lse=l1)
            o2, l2 = pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, descale=inp.descale)
            torch.cuda.synchronize()
            assert not torch.isnan(o1.float()).any() and not torch.isnan(l1).any()
            assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)


@pytest.mark.parametrize("dt", [BF16, FP8])
def test_xcd_grouped_orders_write_every_row(dt):
    # B * Hkv a multiple of 8 turns on the XCD-grouped workgroup orders (query
    # blocks outermost when causal, KV-head groups outermost when not): every
    # output row must still be written exactly as without grouping.
    inp = synth.make_inputs(2, 16, 4, 700, 128, dt, sharp=True, seed=410)
    sc = scale_of(128)
    q, k, v = dev_tensors(inp)
    rows = np.array([0, 699, 700, 5 * 700 + 333, 31 * 700 + 699])
    for causal in (False, True):
        say(f"xcd-grouped order dtype={dt} causal={causal}")
        o = torch.full((2, 16, 700, 128), float("nan"), dtype=torch.bfloat16, device="cuda:0")
        lse = torch.full((2, 16, 700), float("nan"), dtype=torch.float32, device="cuda:0")
        pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=H15, descale=inp.descale, out=o, lse=lse)
        torch.cuda.synchronize()
        assert not torch.isnan(o.float()).any() and not torch.isnan(lse).any()
        o_ref, lse_ref = oracle_run(inp, causal, sc, H15, rows=rows)
        assert_close(inp, o.float().cpu().numpy().astype(np.float64).reshape(-1, 128)[rows],
                     lse.cpu().numpy().astype(np.float64).reshape(-1)[rows], o_ref, lse_ref, "grouped order", H15,
                     causal=causal, sc=sc, rows=rows)


GUARD_SHAPES = [(BF16, 1, 4, 2, 333, 64), (BF16, 1, 4, 2, 333, 128), (FP8, 1, 4, 2, 333, 128),
                (FP8, 2, 3, 3, 129, 64), (BF16, 1, 64, 8, 2500, 128)]  # the last: BF16's 8-wave layout


@pytest.mark.parametrize("dt,B,Hq,Hkv,S,d", GUARD_SHAPES)
def test_writes_stay_inside_outputs(dt, B, Hq, Hkv, S, d):
    # O and LSE as views into larger NaN-filled buffers: every element of the
    # views is written, nothing before or after them is, and the result equals
    # that of a call with outputs of their own (the O rows leave through LDS;
    # the last query block is ragged)
    inp = synth.make_inputs(B, Hq, Hkv, S, d, dt, sharp=True, seed=700 + S + d)
    sc = scale_of(d)
    q, k, v = dev_tensors(inp)
    G = 4096
    n_o, n_l = B * Hq * S * d, B * Hq * S
    for causal in (False, True):
        for mode in (EXACT, H15):
            say(f"guard dtype={dt} shape={(B, Hq, Hkv, S, d)} causal={causal} mode={mode}")
            ob = torch.full((G + n_o + G,), float("nan"), dtype=torch.bfloat16, device="cuda:0")
            lb = torch.full((G + n_l + G,), float("nan"), dtype=torch.float32, device="cuda:0")
            o = ob[G:G + n_o].view(B, Hq, S, d)
            lse = lb[G:G + n_l].view(B, Hq, S)
            pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, descale=inp.descale, out=o, lse=lse)
            o2, l2 = pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, descale=inp.descale)
            torch.cuda.synchronize()
            assert torch.isnan(ob[:G].float()).all() and torch.isnan(ob[G + n_o:].float()).all()
            assert torch.isnan(lb[:G]).all() and torch.isnan(lb[G + n_l:]).all()
            assert not torch.isnan(o.float()).any() and not torch.isnan(lse).any()
            assert torch.equal(o.view(torch.int16), o2.view(torch.int16)) and torch.equal(lse, l2)


EDGE = [(1, 1, 1, 1, 64), (1, 1, 1, 2, 128), (1, 2, 1, 31, 128), (2, 3, 3, 129, 64), (1, 8, 1, 255, 128),
        (3, 4, 2, 257, 128), (1, 16, 2, 1000, 128)]


@pytest.mark.parametrize("B,Hq,Hkv,S,d", EDGE)
@pytest.mark.parametrize("dt", [BF16, FP8])
def test_edge_shapes(B, Hq, Hkv, S, d, dt):
    inp = synth.make_inputs(B, Hq, Hkv, S, d, dt, sharp=False, seed=500 + S)
    sc = scale_of(d)
    for causal in (False, True):
        for mode in ALL_MODES:
            say(f"edge B={B} Hq={Hq} Hkv={Hkv} S={S} d={d} dtype={dt} causal={causal} mode={mode}")
            o, lse = gpu_run(inp, causal, sc, mode)
            o_ref, lse_ref = oracle_run(inp, causal, sc, mode)
            assert_close(inp, o, lse, o_ref, lse_ref, "edge", mode, causal=causal, sc=sc)


def test_side_stream_and_lse_optional():
    inp = synth.make_inputs(1, 4, 4, 384, 128, BF16, sharp=True, seed=600)
    sc = scale_of(128)
    q, k, v = dev_tensors(inp)
    o_ref, l_ref = pkg.attn_fwd(q, k, v, causal=True, scale=sc, exp_mode=H15)
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        o2, _ = pkg.attn_fwd_ex(q, k, v, causal=True, scale=sc, exp_mode=H15, stream=st, want_lse=False)
    st.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(o_ref.view(torch.int16), o2.view(torch.int16))


# ---- Rowmax-PoT (App. A.6 Eq. (rowmax-pot)), BF16 --------------------------

@pytest.mark.parametrize("d,causal,S", [(64, False, 256), (64, True, 300), (128, False, 300), (128, True, 520)])
def test_rowmax_pot_small_full_parity(d, causal, S):
    inp = synth.make_inputs(1, 4, 2, S, d, BF16, sharp=True, seed=800 + S + d)
    sc = scale_of(d)
    say(f"rowmax-pot d={d} causal={causal} S={S}")
    o, lse = gpu_run(inp, causal, sc, POT)
    o_ref, lse_ref = oracle_run(inp, causal, sc, POT)
    assert_close(inp, o, lse, o_ref, lse_ref, "rowmax-pot", POT)


def check_pot_probe(inp, S, causal, sc, rowsets):
    q, k, v = dev_tensors(inp)
    c1 = oracle.c1(sc)
    for (b, h, r0, n) in rowsets:
        say(f"rowmax-pot probe causal={causal} head {h} rows {r0}+{n}")
        o_p, lse_p, s, w, pbits = pkg.attn_fwd_probe(q, k, v, causal=causal, scale=sc, exp_mode=POT, b=b, h=h,
                                                     row0=r0, nrows=n)
        o_m, lse_m = pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=POT)
        torch.cuda.synchronize()
        assert torch.equal(o_p.view(torch.int16), o_m.view(torch.int16)) and torch.equal(lse_p, lse_m)
        s, w, pbits, lse_p = s.cpu().numpy(), w.cpu().numpy(), pbits.cpu().numpy().astype(np.uint32), lse_p.cpu().numpy()
        for r in range(n):
            i = r0 + r
            w_ref, p_ref, lse_ref = oracle.pot_row_from_logits(np.where(np.isneginf(s[r]), np.float32(0), s[r]), i,
                                                                causal, c1)
            assert np.array_equal(w[r].view(np.uint32), w_ref.view(np.uint32)), f"row {i}"
            assert np.array_equal(pbits[r], p_ref), f"row {i}"
            assert abs(lse_p[b, h, i] - lse_ref) <= 1e-5, f"row {i}"


@pytest.mark.parametrize("causal", [False, True])
def test_rowmax_pot_probe_bit_exact(causal):
    S = 520
    inp = synth.make_inputs(1, 4, 1, S, 128, BF16, sharp=True, seed=801)
    check_pot_probe(inp, S, causal, scale_of(128), ((0, 0, 0, 40), (0, 3, 250, 40), (0, 2, S - 37, 37)))


POT_FULL = [synth.WORKLOADS[n] for n in ("causal_bf16_b4_h32kv8_s2048_d128_sharp",
                                         "causal_bf16_b1_h64kv8_s16384_d128_sharp")]


@pytest.mark.parametrize("w", POT_FULL, ids=[w.name for w in POT_FULL])
def test_rowmax_pot_full_size(w):
    say(f"rowmax-pot full-size {w.name}: inputs")
    inp = synth.workload_inputs(w)
    sc = scale_of(w.d)
    tensors = dev_tensors(inp)
    o, lse = gpu_run(inp, w.causal, sc, POT, tensors)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    rng = np.random.default_rng(9)
    nrows_total = w.B * w.Hq * w.S
    rows = np.unique(np.concatenate([[0, w.S - 1, nrows_total - 1], rng.integers(0, nrows_total, 9)]))
    say(f"rowmax-pot full-size {w.name}: oracle on {len(rows)} rows")
    o_ref, lse_ref = oracle_run(inp, w.causal, sc, POT, rows=rows)
    assert_close(inp, o.reshape(-1, w.d)[rows], lse.reshape(-1)[rows], o_ref, lse_ref, "rowmax-pot sampled", POT)
    check_pot_probe(inp, w.S, w.causal, sc, ((w.B - 1, w.Hq - 1, w.S - 40, 40),))


@pytest.mark.parametrize("mode", [EXACT, H15])
def test_attn_fwd_fp8_takes_unit_descales(mode):
    # attn_fwd has no descale arguments: FP8 operands are taken as stored,
    # the same as attn_fwd_ex with descales (1, 1, 1).  The operands are
    # encoded at unit scale (Gaussian values, |x| < 5, as e4m3 codes), so the
    # real logits keep the size the LSE bar assumes; the launcher still takes
    # the FP32 clamp, its exponent bound at unit descales being far above 2^15
    base = synth.make_inputs(1, 4, 2, 300, 128, FP8, sharp=True, seed=990)
    rng = np.random.default_rng(990)
    codes = [synth.e4m3_codes(rng.standard_normal(x.shape).astype(np.float32)) for x in (base.q, base.k, base.v)]
    inp = synth.Inputs(*codes, (1.0, 1.0, 1.0), FP8)
    q, k, v = dev_tensors(inp)
    sc = scale_of(128)
    o1, l1 = pkg.attn_fwd(q, k, v, causal=True, scale=sc, exp_mode=mode)
    o2, l2 = pkg.attn_fwd_ex(q, k, v, causal=True, scale=sc, exp_mode=mode, descale=(1.0, 1.0, 1.0))
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
    unit = synth.Inputs(inp.q, inp.k, inp.v, (1.0, 1.0, 1.0), FP8)
    o_ref, lse_ref = oracle_run(unit, True, sc, mode)
    assert_close(unit, o1.float().cpu().numpy().astype(np.float64), l1.cpu().numpy().astype(np.float64), o_ref,
                 lse_ref, "attn_fwd fp8", mode, causal=True, sc=sc)
