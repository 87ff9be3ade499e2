"""Shared helpers of the GPU parity tests: device copies of the seeded inputs,
GPU and oracle runs, and the comparison bars.

Bars: max |O_gpu - O_oracle| <= 2e-2 max|V| for BF16 operands and 6e-2 max|V|
for FP8 (V dequantised).  LSE: 1e-3 for the exact control.  For the lattice
weights (Rowmax-H15 and S(Q_{2^-k})) compared with the oracle on its own
logits, each row's LSE is held to a bound derived from how far the GPU's
logits may sit from the exact ones (lse_bound_lattice); against the oracle fed
the GPU's own logits, W and P must match bit for bit (check_probe)."""
import math
import sys

import numpy as np
import torch

import oracle
import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth

BF16, FP8 = synth.BF16, synth.FP8_E4M3
EXACT, H15, SQ4, SQ8 = pkg.ATTN_EXP_EXACT, pkg.ATTN_EXP_H15, pkg.ATTN_EXP_SQ4, pkg.ATTN_EXP_SQ8
APPROX = (H15, SQ4, SQ8)
ALL_MODES = (EXACT,) + APPROX
POT = pkg.ATTN_EXP_ROWMAX_POT  # BF16 only
ORACLE_MODE = {EXACT: oracle.EXACT, H15: oracle.H15_TILE, SQ4: oracle.SQ4_TILE, SQ8: oracle.SQ8_TILE,
               POT: oracle.ROWMAX_POT}
ORDER = {H15: 1, SQ4: 2, SQ8: 3}  # input-rounding exponent k
TOL = {BF16: 2e-2, FP8: 6e-2}
LSE_TOL = 1e-3
LSE_TOL_POT = 5e-2
# Accuracy of a GPU logit, relative to sum_c |q_c k_c| of the stored
# operands: the bf16 matrix core accumulates in fp32 (about d 2^-24 = 2^-17
# at d = 128); the fp8 one sums its 64 products less exactly (measured about
# 2^-13).  The probe tests hold the GPU to these.
LOGIT_REL = {BF16: 2.0 ** -16, FP8: 2.0 ** -12}


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_tensors(inp):
    d = torch.device("cuda:0")
    if inp.dtype == BF16:
        return tuple(torch.from_numpy(x.view(np.int16)).to(d).view(torch.bfloat16) for x in (inp.q, inp.k, inp.v))
    return tuple(torch.from_numpy(x).to(d).view(torch.float8_e4m3fn) for x in (inp.q, inp.k, inp.v))


def vmax(inp):
    dec = synth.bf16_decode(inp.v) if inp.dtype == BF16 else synth.e4m3_decode(inp.v) * inp.descale[2]
    return float(np.max(np.abs(dec)))


def scale_of(d):
    return float(np.float32(1.0 / math.sqrt(d)))


def gpu_run(inp, causal, scale, mode, tensors=None):
    q, k, v = tensors if tensors is not None else dev_tensors(inp)
    o, lse = pkg.attn_fwd_ex(q, k, v, causal=causal, scale=scale, exp_mode=mode, descale=inp.descale)
    torch.cuda.synchronize()
    return o.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def oracle_run(inp, causal, scale, mode, rows=None):
    om = ORACLE_MODE[mode]
    return oracle.attn(inp.q, inp.k, inp.v, dtype=inp.dtype, causal=causal, scale=scale, mode=om,
                       descale=inp.descale, Bc=pkg.attn_tile_bc(), rows=rows)


def decoded(x, dt):
    return np.asarray(synth.bf16_decode(x) if dt == BF16 else synth.e4m3_decode(x), np.float64)


def stratified_rows(B, Hq, S, br, seed):
    """Flat row indices (b * Hq + h) * S + i for a full-size check: one row of
    every (b, h), whose wave slot within its workgroup (br rows, 32 per wave)
    cycles over the heads; the first and last row of query blocks of four
    heads; the tensor's first and last row."""
    rng = np.random.default_rng(seed)
    nw, nqb = br // 32, (S + br - 1) // br
    rows = []
    for j in range(B * Hq):  # every (b, h); wave slots cycle over the heads
        qb = int(rng.integers(nqb))
        i = min(qb * br + 32 * (j % nw) + int(rng.integers(32)), S - 1)
        rows.append(j * S + i)
    for j in rng.choice(B * Hq, min(4, B * Hq), replace=False):  # first and last row of query blocks
        qb = int(rng.integers(nqb))
        rows += [int(j) * S + qb * br, int(j) * S + min(qb * br + br - 1, S - 1)]
    rows += [0, B * Hq * S - 1]
    return np.unique(np.array(rows, np.int64))


def lse_bound_lattice(s, qrow, krows, jend, i, causal, c1, dt, k, Bc, lse_ref):
    """Bound on |LSE_gpu - LSE_oracle| of one row for a lattice weight, the
    oracle on its own logits s (fp32, exact dot products rounded once) and
    the GPU on logits within e_j = LOGIT_REL sum_c |q_c k_jc| + 2^-24 |s_j| of
    them.  (qrow, krows: the stored operand values, without descales.)

    A logit moved by e moves y = 2^k c1 (s - m) + 2^k off by at most
    2^k c1 (e_j + e_a), e_a bounding the move of the running maximum m of
    key j's tile: the GPU's maximum can only come from a key within 2 max e
    of that maximum, so e_a is the largest e among those keys.  A lattice
    weight changes only where y crosses a rounding boundary (a half-integer),
    and then by at most half of itself (adjacent lattice values differ by a
    factor 1.5 or 4/3).  Moving the anchors by at most e_a moves LSE by
    ln2 c1 max e_a when no weight changes.  So |dLSE| <= ln2 c1 max e_a -
    ln(1 - sum over keys within reach of a boundary of half their share of
    l), plus the fp32 summation and rescale error of the GPU's l
    ((3 tiles + 64) 2^-24) and four fp32 ulps of the stored LSE."""
    y, anchor, w = oracle.row_exponents_from_logits(s, i, causal, c1, dt, Bc, k=k)
    y, anchor, w = y[:jend].astype(np.float64), anchor[:jend].astype(np.float64), w[:jend].astype(np.float64)
    sv = s[:jend].astype(np.float64)
    e = LOGIT_REL[dt] * (np.abs(krows[:jend]) @ np.abs(qrow)) + 2.0 ** -24 * np.abs(sv)
    reach_m = 2.0 * float(np.max(e))
    e_a = np.zeros(jend)
    for t0 in range(0, jend, Bc):
        t1 = min(t0 + Bc, jend)
        cand = sv[:t1] >= anchor[t0] - reach_m  # keys that may hold the GPU's running max
        e_a[t0:t1] = float(np.max(e[:t1][cand]))
    e_m = float(np.max(e_a))
    dy = 2.0 ** k * c1 * (e + e_a) + 2.0 * np.spacing(np.abs(y).astype(np.float32)).astype(np.float64)
    dist = np.abs(y - (np.floor(y) + 0.5))
    reach = dist <= dy
    share = w * np.exp2(c1 * (anchor - np.max(anchor)))
    share = share / share.sum()
    moved = 0.5 * float(np.sum(share[reach]))
    tiles = (jend + Bc - 1) // Bc
    return (math.log(2) * c1 * e_m - math.log1p(-min(moved, 0.999)) + (3 * tiles + 64) * 2.0 ** -24
            + 4.0 * float(np.spacing(np.float32(abs(lse_ref)))) + 1e-6)


# the constant terms of lse_bound_lattice for one tile (no ulps)
LSE_FLOOR = 67 * 2.0 ** -24 + 1e-6


def lse_bounds(inp, rows, causal, sc, mode):
    """lse_bound_lattice for each flat row (b * Hq + h) * S + i of a square problem."""
    B, Hq, S, d = inp.q.shape
    G = Hq // inp.k.shape[1]
    c1 = oracle.c1(sc, inp.descale[0], inp.descale[1])
    qdec, kdec = decoded(inp.q, inp.dtype), decoded(inp.k, inp.dtype)
    out = np.zeros(len(rows))
    for n, flat in enumerate(rows):
        b, h, i = int(flat) // (Hq * S), (int(flat) // S) % Hq, int(flat) % S
        s = oracle.logits_row(inp.q, inp.k, inp.dtype, b, h, i)
        jend = i + 1 if causal else S
        _, _, l_ref = oracle.sq_row_from_logits(s, i, causal, c1, inp.dtype, pkg.attn_tile_bc(), k=ORDER[mode])
        out[n] = lse_bound_lattice(s, qdec[b, h, i], kdec[b, h // G], jend, i, causal, c1, inp.dtype, ORDER[mode],
                                   pkg.attn_tile_bc(), l_ref)
    return out


def assert_close(inp, o, lse, o_ref, lse_ref, what, mode=EXACT, causal=None, sc=None, rows=None, flat_lse=False):
    """O within the dtype's bar of max|V|; LSE within 1e-3 (exact control),
    within each row's lse_bound_lattice (lattice weights; needs causal, sc
    and the flat row indices, all rows when None), or 5e-2 (Rowmax-PoT, and
    with flat_lse the lattice weights under a nonzero rescale threshold, for
    which the anchors, and so the bound's exponents, differ).
    Every LSE bar also allows four fp32 ulps of |LSE|, the stored value's own
    rounding, which exceeds 1e-5 once |LSE| is in the thousands."""
    o = np.asarray(o).reshape(-1, o.shape[-1])
    o_ref = np.asarray(o_ref).reshape(o.shape)
    lse, lse_ref = np.asarray(lse).reshape(-1), np.asarray(lse_ref).reshape(-1)
    err = float(np.max(np.abs(o - o_ref)))
    dl_raw = np.abs(lse - lse_ref)
    dl = np.maximum(dl_raw - 4.0 * np.spacing(np.abs(lse_ref).astype(np.float32)), 0.0)
    bound = TOL[inp.dtype] * vmax(inp)
    say(f"  {what}: max|dO| {err:.3e} (bound {bound:.3e})  max|dLSE| {float(np.max(dl)):.3e}  "
        f"rows |dLSE|>1e-4: {np.mean(dl > 1e-4):.4f}")
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(lse))
    assert err <= bound, what
    if mode in APPROX and not flat_lse:
        assert causal is not None and sc is not None, "the lattice LSE bound needs the mask and the scale"
        if rows is None:
            rows = np.arange(lse.shape[0])
        rows = np.asarray(rows)
        # every row's bound is at least its constant terms ((3 + 64) 2^-24 +
        # 1e-6 + four ulps of |LSE|); rows that agree that closely pass
        # whatever their bound, so it is computed only for the others
        lb = LSE_FLOOR + 4.0 * np.spacing(np.abs(lse_ref).astype(np.float32)).astype(np.float64)
        above = dl_raw > lb
        if np.any(above):
            lb[above] = lse_bounds(inp, rows[above], causal, sc, mode)
        worst = int(np.argmax(dl_raw - lb))
        say(f"  {what}: LSE within the per-row bound ({int(np.sum(above))} of {len(rows)} rows above its floor, "
            f"worst margin {float(lb[worst] - dl_raw[worst]):.2e})")
        assert np.all(dl_raw <= lb), f"{what}: row {rows[worst]} |dLSE| {dl_raw[worst]:.3e} > {lb[worst]:.3e}"
        # the bound takes every weight within reach to move the same way; in
        # practice they move both ways and rarely: the median row agrees to 1e-4
        assert float(np.median(dl)) <= 1e-4, what
    elif mode == POT or mode in APPROX:
        assert float(np.median(dl)) <= 1e-4 and float(np.max(dl)) <= LSE_TOL_POT, what
    else:
        assert float(np.max(dl)) <= LSE_TOL, what


def check_probe(inp, S, d, dt, causal, mode, sc, rowsets, tensors=None):
    """Probe rows of the kernel: logits close to the exact dot products, and W,
    P and LSE bit-identical (to 1e-5 for LSE) to the oracle fed those logits."""
    q, k, v = tensors if tensors is not None else dev_tensors(inp)
    c1 = oracle.c1(sc, inp.descale[0], inp.descale[1])
    G = inp.q.shape[1] // inp.k.shape[1]
    for (b, h, r0, n) in rowsets:
        say(f"probe dtype={dt} causal={causal} mode={mode} rows {r0}+{n} head ({b},{h})")
        o_p, lse_p, s, w, pbits = pkg.attn_fwd_probe(q, k, v, causal=causal, scale=sc, exp_mode=mode,
                                                     b=b, h=h, row0=r0, nrows=n, descale=inp.descale)
        o_m, lse_m = pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, descale=inp.descale)
        torch.cuda.synchronize()
        # the probe runs the same arithmetic as the timed kernel
        assert torch.equal(o_p.view(torch.int16), o_m.view(torch.int16))
        assert torch.equal(lse_p, lse_m)
        del o_p, o_m, lse_m
        s, w, pbits = s.cpu().numpy(), w.cpu().numpy(), pbits.cpu().numpy().astype(np.uint32)
        lse_p = lse_p[b, h, r0:r0 + n].cpu().numpy()
        qv = decoded(inp.q[b, h, r0:r0 + n], dt)
        kv = decoded(inp.k[b, h // G], dt)
        for r in range(n):
            i = r0 + r
            jend = i + 1 if causal else S
            # GPU logits agree with the exact dot products to within the MFMA's
            # accumulation error (LOGIT_REL of sum_c |q_c k_c|)
            s_ref = oracle.logits_row(inp.q, inp.k, dt, b, h, i)
            mag = np.abs(kv[:jend]) @ np.abs(qv[r])
            assert np.all(np.isneginf(s[r, jend:]))
            rel = np.max(np.abs(s[r, :jend] - s_ref[:jend]) / np.maximum(mag, 1e-30))
            if r == 0:
                say(f"  logit error / sum|q k|: {rel:.3e}")
            assert rel <= LOGIT_REL[dt]
            if mode in APPROX:
                w_ref, p_ref, lse_ref = oracle.sq_row_from_logits(s[r], i, causal, c1, dt, pkg.attn_tile_bc(),
                                                                  k=ORDER[mode])
                # LSE is an fp32 value formed from m c1 + log2 l: at large
                # logits (|LSE| in the thousands) a few of its ulps exceed 1e-5.
                # l itself is an fp32 sum of positive weights, one add per key
                # tile into the running sum after in-tile partial sums, so its
                # relative error is bounded by (tiles + 64) 2^-24; that bound
                # passes 1e-5 beyond about 104 tiles (13K keys).
                sum_bound = (jend / pkg.attn_tile_bc() + 64) * 2.0 ** -24
                lse_tol = max(1e-5, 4.0 * float(np.spacing(np.float32(abs(lse_ref))))) + sum_bound
                assert abs(lse_p[r] - lse_ref) <= lse_tol, f"row {i}"
                assert np.array_equal(w[r].view(np.uint32), w_ref.view(np.uint32)), f"row {i}"
                assert np.array_equal(pbits[r], p_ref), f"row {i}"
            else:
                w_ref, _, _ = oracle.h15_row_from_logits(s[r], i, causal, c1, dt, pkg.attn_tile_bc(), exact_exp=True)
                # hardware exp2 (about 1 ulp); P is the stored rounding of the GPU's own w
                assert np.max(np.abs(w[r] - w_ref) / np.maximum(w_ref, 1e-30)) < 4e-7
                wb = w[r].view(np.uint32).astype(np.uint64)
                enc = (((wb + 0x7FFF + ((wb >> 16) & 1)) >> 16).astype(np.uint32) if dt == BF16
                       else np.array([oracle.e4m3_encode(float(x)) for x in w[r]], np.uint32))
                assert np.array_equal(pbits[r], enc), f"row {i}"
