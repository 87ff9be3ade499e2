"""The stratified row sample of the full-size GPU checks (parity_helpers.
stratified_rows), checked on the CPU for every workload shape and every
shape of the parity grid: valid flat indices, one row of every (batch,
head), every wave slot of a workgroup hit when there are at least as many
heads as wave slots, first and last rows of query blocks, and the tensor's
first and last row."""
import numpy as np
import pytest

from paper_2609_33586_amd import synth
from parity_helpers import stratified_rows

SHAPES = sorted({(w.B, w.Hq, w.S, 256 if w.dtype == synth.BF16 else 128) for w in synth.WORKLOADS.values()}
                | {(B, Hq, S, br) for (S, (B, Hq)) in ((2048, (4, 32)), (8192, (2, 32)), (16384, (1, 64)))
                   for br in (128, 256)}
                | {(1, 1, 1, 128), (1, 1, 300, 256), (1, 3, 129, 128)})


@pytest.mark.parametrize("B,Hq,S,br", SHAPES)
def test_stratified_rows(B, Hq, S, br):
    rows = stratified_rows(B, Hq, S, br, seed=7)
    assert rows.dtype == np.int64 and np.all(np.diff(rows) > 0)
    assert rows[0] == 0 and rows[-1] == B * Hq * S - 1
    assert np.all((rows >= 0) & (rows < B * Hq * S))
    heads, pos = rows // S, rows % S
    assert set(heads.tolist()) == set(range(B * Hq))  # every (b, h)
    nw = br // 32
    slots = {int(p % br) // 32 for p in pos}
    if B * Hq >= nw and S >= br:
        assert slots == set(range(nw))  # every wave slot of a workgroup
    starts = [p for p in pos if p % br == 0]
    ends = [p for p in pos if p % br == br - 1 or p == S - 1]
    assert starts and ends  # first and last rows of query blocks
