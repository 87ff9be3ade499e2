"""GPU parity over the grid of App. B.3's latency table: sequence lengths
2K, 8K and 16K, causal and non-causal, BF16 and FP8 operands, the exact
control and Rowmax-H15, at the GQA shapes of the full-size workloads
(B4 Hq32 Hkv8 at 2K, B2 Hq32 Hkv8 at 8K, B1 Hq64 Hkv8 at 16K; d = 128, 2%
sharp keys).

Each cell runs the kernel once on NaN-filled outputs, then checks:
  * every output row was written and is finite, and |O| <= max|V| (O is a
    convex combination of V rows);
  * stratified rows against the oracle (parity_helpers bars): one row of
    every (batch, head), cycling through every wave slot of a workgroup; the
    first and last row of query blocks; the tensor's first and last row;
  * 40 probe rows across a query-block boundary, bit-exact W and P against
    the oracle fed the GPU's own logits."""
import numpy as np
import pytest
import torch

import paper_2609_33586_amd as pkg
from paper_2609_33586_amd import synth
from parity_helpers import (BF16, EXACT, FP8, H15, assert_close, check_probe, dev_tensors, oracle_run, say,
                            scale_of, stratified_rows, vmax)

pytestmark = pytest.mark.gpu

SHAPES = {2048: (4, 32, 8), 8192: (2, 32, 8), 16384: (1, 64, 8)}  # S: (B, Hq, Hkv)
D = 128
# query rows per workgroup: 8 waves of 32 rows (BF16), 4 waves (FP8)
BR = {BF16: 256, FP8: 128}
CELLS = [(S, dt, causal, mode) for S in SHAPES for dt in (BF16, FP8) for causal in (False, True)
         for mode in (EXACT, H15)]

_cache = {}


def inputs(S, dt):
    key = (S, dt)
    if key not in _cache:
        _cache.clear()
        torch.cuda.empty_cache()
        B, Hq, Hkv = SHAPES[S]
        say(f"grid inputs S={S} dtype={dt}: generating")
        inp = synth.make_inputs(B, Hq, Hkv, S, D, dt, sharp=True, seed=3000 + S // 1024 + 100 * dt)
        _cache[key] = (inp, dev_tensors(inp))
    return _cache[key]


@pytest.mark.parametrize("S,dt,causal,mode", CELLS,
                         ids=[f"S{S}-{'bf16' if dt == BF16 else 'fp8'}-{'causal' if c else 'noncausal'}-"
                              f"{'exact' if m == EXACT else 'h15'}" for S, dt, c, m in CELLS])
def test_grid_cell(S, dt, causal, mode):
    inp, tensors = inputs(S, dt)
    q, k, v = tensors
    B, Hq, Hkv = SHAPES[S]
    sc = scale_of(D)
    say(f"grid S={S} dtype={dt} causal={causal} mode={mode}: GPU run")
    o = torch.full((B, Hq, S, D), float("nan"), dtype=torch.bfloat16, device=q.device)
    lse = torch.full((B, Hq, S), float("nan"), dtype=torch.float32, device=q.device)
    pkg.attn_fwd_ex(q, k, v, causal=causal, scale=sc, exp_mode=mode, descale=inp.descale, out=o, lse=lse)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(lse).all()), "an LSE row was not written"
    omax = float(o.float().abs().amax())  # NaN propagates: an unwritten O row fails here
    assert omax <= vmax(inp) * (1 + 2 ** -7), omax
    rows = stratified_rows(B, Hq, S, BR[dt], seed=S + 10 * dt + 100 * causal + 1000 * mode)
    rows_t = torch.from_numpy(rows).to(q.device)
    o_rows = o.view(-1, D)[rows_t].float().cpu().numpy().astype(np.float64)
    lse_rows = lse.view(-1)[rows_t].cpu().numpy().astype(np.float64)
    del o, lse
    say(f"grid S={S} dtype={dt} causal={causal} mode={mode}: oracle on {len(rows)} rows")
    o_ref, lse_ref = oracle_run(inp, causal, sc, mode, rows=rows)
    assert_close(inp, o_rows, lse_rows, o_ref, lse_ref, "stratified rows", mode, causal=causal, sc=sc, rows=rows)
    # 40 probe rows across the middle query-block boundary of one head
    b, h = B - 1, (S // 1024 + 3 * dt) % Hq
    check_probe(inp, S, D, dt, causal, mode, sc, ((b, h, S // 2 - 20, 40),), tensors)
