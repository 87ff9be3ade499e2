"""The per-row LSE bar that the GPU parity tests apply to the lattice weights
(parity_helpers.lse_bound_lattice), checked on the CPU: logits moved by at
most the error the bar assumes for the GPU's matrix core (random moves, and
moves chosen to push every weight within reach across its rounding
boundary) must change the oracle's LSE by no more than the bound."""
import numpy as np
import pytest

import oracle
from paper_2609_33586_amd import synth
from parity_helpers import LOGIT_REL, decoded, lse_bound_lattice

BC = 128


@pytest.mark.parametrize("dt", [synth.BF16, synth.FP8_E4M3])
@pytest.mark.parametrize("k", [1, 2, 3])
@pytest.mark.parametrize("causal", [False, True])
def test_bound_holds_for_moved_logits(dt, k, causal):
    S, d = 700, 128
    inp = synth.make_inputs(1, 2, 1, S, d, dt, sharp=True, seed=880 + k)
    sc = float(np.float32(1 / np.sqrt(d)))
    c1 = oracle.c1(sc, inp.descale[0], inp.descale[1])
    qdec, kdec = decoded(inp.q, dt), decoded(inp.k, dt)
    rng = np.random.default_rng(881)
    bounds = []
    for i in (0, 127, 128, 450, S - 1):
        s = oracle.logits_row(inp.q, inp.k, dt, 0, 1, i)
        jend = i + 1 if causal else S
        _, _, l_ref = oracle.sq_row_from_logits(s, i, causal, c1, dt, BC, k=k)
        bound = lse_bound_lattice(s, qdec[0, 1, i], kdec[0, 0], jend, i, causal, c1, dt, k, BC, l_ref)
        bounds.append(bound)
        e = LOGIT_REL[dt] * (np.abs(kdec[0, 0, :jend]) @ np.abs(qdec[0, 1, i]))
        y, _, _ = oracle.row_exponents_from_logits(s, i, causal, c1, dt, BC, k=k)
        # push each logit by its full allowance toward its nearest rounding
        # boundary, then the other way, then at random
        toward = np.sign((np.floor(y[:jend]) + 0.5) - y[:jend])
        for move in (toward * e, -toward * e, rng.uniform(-1, 1, jend) * e):
            s2 = s.copy()
            s2[:jend] = (s[:jend].astype(np.float64) + move).astype(np.float32)
            _, _, l2 = oracle.sq_row_from_logits(s2, i, causal, c1, dt, BC, k=k)
            assert abs(l2 - l_ref) <= bound, (i, abs(l2 - l_ref), bound)
    print(f"bounds: {[f'{b:.2e}' for b in bounds]}")
    # BF16: tighter than the flat 5e-2 used before, for every row here.  (At
    # FP8 the 2^-12 logit allowance puts more keys within reach of a
    # boundary, the more so for the finer roundings k = 2, 3.)
    if dt == synth.BF16:
        assert max(bounds) < 5e-2
